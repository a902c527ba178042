"""Plain fp64 CPU oracle for the SENSE retrieval + soft-gated evaluation path.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, ``__graft_entry__.smoke()``
and the benchmark's ``cpu_baseline`` leg may import this package.  The HIP
library never imports, links or calls it, and it imports nothing from the HIP
library (the two share no code).

The arithmetic lives in ``sense_oracle.c`` (plain C loops in double precision;
see its header for the paper passages it follows and the readings taken) and,
for the loose trie of Alg. 3, in ``trie.py`` (plain numpy).  This module
marshals numpy arrays into the C library through ctypes.

Array conventions: float32 data is passed as ``np.float32`` arrays; binary16
and bfloat16 data are passed as ``np.uint16`` arrays of raw bit patterns with
``dtype='f16'`` or ``dtype='bf16'``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sense_oracle.c")
_LIB = os.path.join(_HERE, "libsense_oracle.so")

DTYPES = {"f32": 0, "f16": 1, "bf16": 2}
METRICS = {"ip": 0, "cosine": 1}


def build(force: bool = False) -> str:
    """Compile the oracle with the host C compiler (OpenMP over rows).  The
    environment variable SENSE_ORACLE_LIB names a library built elsewhere
    (the sanitizer and planted-mistake checks of the test-suite) to load
    instead."""
    alt = os.environ.get("SENSE_ORACLE_LIB")
    if alt:
        return alt
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", _SRC, "-o", tmp, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        P, I32, I64, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.oracle_decode_f16.argtypes = [ctypes.c_uint16]
        lib.oracle_decode_f16.restype = D
        lib.oracle_decode_bf16.argtypes = [ctypes.c_uint16]
        lib.oracle_decode_bf16.restype = D
        lib.oracle_scores.argtypes = [P, ctypes.c_int, I64, I32, I64, P, ctypes.c_int, I32, ctypes.c_int, P]
        lib.oracle_topk.argtypes = [P, I64, I32, P, P]
        lib.oracle_gather.argtypes = [P, P, I32, P, I32, P, P]
        lib.oracle_row_stats.argtypes = [P, ctypes.c_int, I32, I32, P, P, P]
        lib.oracle_soft_gate_verify.argtypes = [
            P, ctypes.c_int, I64, P, P, I32, I32, I32, I32, D, I32, I32, I32, I32, P, P, P, P, P, P
        ]
        lib.oracle_select_candidates.argtypes = [P, P, P, I32, P, P, P, I32, I32, I32, I32, D, D,
                                                 D, I32, I32, P, P, P, P]
        lib.oracle_project.argtypes = [P, ctypes.c_int, I64, I32, I64, P, P, I32, I32, P]
        lib.oracle_ivf_assign.argtypes = [P, ctypes.c_int, I64, I32, I64, P, I32, ctypes.c_int, P, P]
        lib.oracle_pq_encode.argtypes = [P, ctypes.c_int, I64, I32, I64, P, P, P, I32, I32, P]
        lib.oracle_ivf_search.argtypes = [P, I32, P, I32, ctypes.c_int, I32, P, I64, P,
                                          ctypes.c_int, I64, P, P, I32, I32, I32, P, P, P, P]
        for f in ("oracle_scores", "oracle_topk", "oracle_gather", "oracle_row_stats",
                  "oracle_soft_gate_verify", "oracle_select_candidates", "oracle_project",
                  "oracle_ivf_assign", "oracle_pq_encode", "oracle_ivf_search"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def set_threads(n: int) -> int:
    """Threads the oracle's OpenMP loops use from now on (the host baseline is
    timed on all cores and on one); returns the previous count."""
    lib = _load()
    lib.omp_get_max_threads.restype = ctypes.c_int
    lib.omp_set_num_threads.argtypes = [ctypes.c_int]
    prev = int(lib.omp_get_max_threads())
    lib.omp_set_num_threads(int(n))
    return prev


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _raw(a, dtype):
    want = np.float32 if dtype == "f32" else np.uint16
    a = np.ascontiguousarray(a)
    if a.dtype != want:
        raise TypeError(f"dtype {dtype} wants {want}, got {a.dtype}")
    return a


def decode(bits, dtype: str) -> np.ndarray:
    """Decode raw f16/bf16 bit patterns (or pass f32 through) to float64."""
    lib = _load()
    if dtype == "f32":
        return np.asarray(bits, dtype=np.float32).astype(np.float64)
    fn = lib.oracle_decode_f16 if dtype == "f16" else lib.oracle_decode_bf16
    flat = np.asarray(bits, dtype=np.uint16).ravel()
    return np.array([fn(int(b)) for b in flat], dtype=np.float64).reshape(np.shape(bits))


def scores(keys, key_dtype: str, queries, q_dtype: str, metric: str = "cosine",
           key_stride: int | None = None, d: int | None = None) -> np.ndarray:
    """Exact similarity of every query to every key row: (Q, N) float64."""
    keys = _raw(keys, key_dtype)
    queries = _raw(queries, q_dtype)
    n = keys.shape[0]
    stride = keys.shape[1] if key_stride is None else key_stride
    d = stride if d is None else d
    q2 = queries.reshape(-1, d)
    out = np.empty((q2.shape[0], n), dtype=np.float64)
    rc = _load().oracle_scores(_ptr(keys), DTYPES[key_dtype], n, d, stride, _ptr(q2),
                               DTYPES[q_dtype], q2.shape[0], METRICS[metric], _ptr(out))
    if rc:
        raise ValueError("oracle_scores rejected its arguments")
    return out


def topk(score_row: np.ndarray, k: int):
    """Full sort by (score desc, index asc); first k (ids int64, scores f64)."""
    s = np.ascontiguousarray(score_row, dtype=np.float64)
    ids = np.empty(k, dtype=np.int64)
    sc = np.empty(k, dtype=np.float64)
    if _load().oracle_topk(_ptr(s), s.shape[0], k, _ptr(ids), _ptr(sc)):
        raise ValueError("oracle_topk rejected its arguments")
    return ids, sc


def gather(spans: np.ndarray, span_len, ids: np.ndarray):
    """Candidate draft batch of the given hits: (drafts[k, M] int32, len[k])."""
    spans = np.ascontiguousarray(spans, dtype=np.int32)
    max_span = spans.shape[1]
    sl = None if span_len is None else np.ascontiguousarray(span_len, dtype=np.int32)
    ids = np.ascontiguousarray(ids, dtype=np.int64)
    k = ids.shape[0]
    drafts = np.empty((k, max_span), dtype=np.int32)
    dl = np.empty(k, dtype=np.int32)
    if _load().oracle_gather(_ptr(spans), _ptr(sl), max_span, _ptr(ids), k, _ptr(drafts), _ptr(dl)):
        raise ValueError("oracle_gather rejected its arguments")
    return drafts, dl


def retrieve(keys, key_dtype, queries, q_dtype, k, spans, span_len=None, metric="cosine"):
    """Exact retrieval: per query the top-k (ids, scores) and gathered drafts."""
    s = scores(keys, key_dtype, queries, q_dtype, metric)
    out_ids, out_sc, out_dr, out_dl = [], [], [], []
    for q in range(s.shape[0]):
        ids, sc = topk(s[q], k)
        dr, dl = gather(spans, span_len, ids)
        out_ids.append(ids); out_sc.append(sc); out_dr.append(dr); out_dl.append(dl)
    return np.stack(out_ids), np.stack(out_sc), np.stack(out_dr), np.stack(out_dl)


def row_stats(row, dtype: str, tok: int):
    """(argmax, entropy in nats, rank of tok) of one logit row."""
    row = _raw(row, dtype)
    y = ctypes.c_int32()
    e = ctypes.c_double()
    r = ctypes.c_int32()
    if _load().oracle_row_stats(_ptr(row), DTYPES[dtype], row.shape[-1], tok,
                                ctypes.byref(y), ctypes.byref(e), ctypes.byref(r)):
        raise ValueError("oracle_row_stats rejected its arguments")
    return y.value, e.value, r.value


def soft_gate_verify(logits, dtype: str, drafts, draft_len=None, n_groups: int = 1,
                     gamma: float = 0.05, topk: int = 3, window: int = 6, tau: int = 0,
                     entropy_normalized: bool = True, vocab: int | None = None):
    """Alg. 4 literally.  logits: (C, M, stride) array; drafts: (C, M) int32.

    Returns a dict with accept_len (C,), best (n_groups,), gate_score (C, M),
    masks (C, M) uint8, argmax (C, M), rank (C, M)."""
    logits = _raw(logits, dtype)
    drafts = np.ascontiguousarray(drafts, dtype=np.int32)
    c, m = drafts.shape
    stride = logits.shape[-1]
    v = stride if vocab is None else vocab
    dl = None if draft_len is None else np.ascontiguousarray(draft_len, dtype=np.int32)
    acc = np.empty(c, dtype=np.int32)
    best = np.empty(max(n_groups, 1), dtype=np.int32)
    gs = np.empty((c, m), dtype=np.float64)
    masks = np.empty((c, m), dtype=np.uint8)
    am = np.empty((c, m), dtype=np.int32)
    rk = np.empty((c, m), dtype=np.int32)
    rc = _load().oracle_soft_gate_verify(
        _ptr(logits), DTYPES[dtype], stride, _ptr(drafts), _ptr(dl), c, m, v, n_groups,
        float(gamma), topk, window, tau, int(bool(entropy_normalized)),
        _ptr(acc), _ptr(best), _ptr(gs), _ptr(masks), _ptr(am), _ptr(rk))
    if rc:
        raise ValueError("oracle_soft_gate_verify rejected its arguments")
    return {"accept_len": acc, "best": best[:n_groups], "gate_score": gs, "masks": masks,
            "argmax": am, "rank": rk}


def select_candidates(scores_s, drafts_s, len_s, anchor: int, top_n: int, alpha: float,
                      beta: float, delta: float = 0.0, anchor_override: bool = True,
                      scores_d=None, drafts_d=None, len_d=None, precision: str = "f64"):
    """Composite-score Top-N over static + dynamic hits with the anchor
    override (Sec. 3.2 Eq. 8, Alg. 2).  Returns (drafts, lengths, source,
    composite scores).  precision "f32" takes the composite score in binary32
    (delta added in binary32, one fused multiply-add)."""
    def prep(sc, dr, ln):
        if sc is None:
            return None, None, None, 0
        sc = np.ascontiguousarray(sc, dtype=np.float64)
        dr = np.ascontiguousarray(dr, dtype=np.int32)
        ln = None if ln is None else np.ascontiguousarray(ln, dtype=np.int32)
        return sc, dr, ln, sc.shape[0]
    ss, ds, ls, ns = prep(scores_s, drafts_s, len_s)
    sd, dd, ld, nd = prep(scores_d, drafts_d, len_d)
    m = (ds if ds is not None else dd).shape[1]
    out_dr = np.empty((top_n, m), dtype=np.int32)
    out_len = np.empty(top_n, dtype=np.int32)
    out_src = np.empty(top_n, dtype=np.int32)
    out_sc = np.empty(top_n, dtype=np.float64)
    rc = _load().oracle_select_candidates(
        _ptr(ss), _ptr(ds), _ptr(ls), ns, _ptr(sd), _ptr(dd), _ptr(ld), nd, int(anchor), m,
        top_n, float(alpha), float(beta), float(delta), int(bool(anchor_override)),
        {"f64": 0, "f32": 1}[precision], _ptr(out_dr), _ptr(out_len), _ptr(out_src), _ptr(out_sc))
    if rc:
        raise ValueError("oracle_select_candidates rejected its arguments")
    return out_dr, out_len, out_src, out_sc


def project(x, x_dtype: str, basis, mean=None, normalize: bool = True,
            x_stride: int | None = None, d_in: int | None = None) -> np.ndarray:
    """PCA projection + optional L2 normalisation of the rows of x (Alg. 2's
    L2Norm(PCA(h)); the datastore projection Z): (n, d_out) float64.  basis
    is d_out x d_in (principal directions as rows), mean d_in or None."""
    x = _raw(x, x_dtype)
    basis = np.ascontiguousarray(basis, dtype=np.float64)
    d_out, din = basis.shape
    d_in = din if d_in is None else d_in
    stride = x.shape[-1] if x_stride is None else x_stride
    n = x.size // stride
    mean = None if mean is None else np.ascontiguousarray(mean, dtype=np.float64)
    out = np.empty((n, d_out), dtype=np.float64)
    rc = _load().oracle_project(_ptr(x), DTYPES[x_dtype], n, d_in, stride, _ptr(mean),
                                _ptr(basis), d_out, int(bool(normalize)), _ptr(out))
    if rc:
        raise ValueError("oracle_project rejected its arguments")
    return out


def ivf_assign(keys, key_dtype: str, centroids, metric: str = "cosine"):
    """List of every key (most similar centroid, ties lower id) and that
    similarity: (lists int32 [n], scores float64 [n])."""
    keys = _raw(keys, key_dtype)
    n, d = keys.shape
    cen = np.ascontiguousarray(centroids, dtype=np.float64)
    lists = np.empty(n, dtype=np.int32)
    sc = np.empty(n, dtype=np.float64)
    if _load().oracle_ivf_assign(_ptr(keys), DTYPES[key_dtype], n, d, d, _ptr(cen), cen.shape[0],
                                 METRICS[metric], _ptr(lists), _ptr(sc)):
        raise ValueError("oracle_ivf_assign rejected its arguments")
    return lists, sc


def pq_encode(keys, key_dtype: str, centroids, lists, codebooks):
    """PQ codes (n x m uint8) of the residuals key - centroid[list];
    codebooks is m x ksub x dsub."""
    keys = _raw(keys, key_dtype)
    n, d = keys.shape
    cen = np.ascontiguousarray(centroids, dtype=np.float64)
    lists = np.ascontiguousarray(lists, dtype=np.int32)
    cb = np.ascontiguousarray(codebooks, dtype=np.float64)
    m, ksub, _ = cb.shape
    codes = np.empty((n, m), dtype=np.uint8)
    if _load().oracle_pq_encode(_ptr(keys), DTYPES[key_dtype], n, d, d, _ptr(cen), _ptr(lists),
                                _ptr(cb), m, ksub, _ptr(codes)):
        raise ValueError("oracle_pq_encode rejected its arguments")
    return codes


def ivf_search(query, centroids, lists, nprobe: int, k: int, metric: str = "cosine",
               keys=None, key_dtype: str = "bf16", codes=None, codebooks=None):
    """IVF-Flat (keys given) or IVF-PQ (codes and codebooks given) search of
    one fp64 query.  Returns (probe [nprobe] int32, coarse [nlist] float64,
    ids [k] int64, scores [k] float64)."""
    q = np.ascontiguousarray(query, dtype=np.float64).ravel()
    cen = np.ascontiguousarray(centroids, dtype=np.float64)
    nlist, d = cen.shape
    lists = np.ascontiguousarray(lists, dtype=np.int32)
    n = lists.shape[0]
    kk = None if keys is None else _raw(keys, key_dtype)
    cd = None if codes is None else np.ascontiguousarray(codes, dtype=np.uint8)
    cb = None if codebooks is None else np.ascontiguousarray(codebooks, dtype=np.float64)
    m, ksub = (cb.shape[0], cb.shape[1]) if cb is not None else (0, 0)
    probe = np.empty(nprobe, dtype=np.int32)
    coarse = np.empty(nlist, dtype=np.float64)
    ids = np.empty(k, dtype=np.int64)
    sc = np.empty(k, dtype=np.float64)
    rc = _load().oracle_ivf_search(_ptr(q), d, _ptr(cen), nlist, METRICS[metric], nprobe,
                                   _ptr(lists), n, _ptr(kk), DTYPES[key_dtype], d, _ptr(cd),
                                   _ptr(cb), m, ksub, k, _ptr(probe), _ptr(coarse), _ptr(ids),
                                   _ptr(sc))
    if rc:
        raise ValueError("oracle_ivf_search rejected its arguments")
    return probe, coarse, ids, sc


def dynamic_spans(tokens, max_span: int):
    """Continuation table of a dynamic context cache (Alg. 1's retriever
    update; Alg. 2's dynamic search): the key stored at position p predicted
    token p, so its continuation is tokens[p : p + max_span], cut at the end
    of what has been generated.  Returns (spans n x max_span int32 padded
    with -1, lengths n int32)."""
    tokens = np.asarray(tokens, dtype=np.int32)
    n = tokens.shape[0]
    spans = np.full((n, max_span), -1, dtype=np.int32)
    lens = np.empty(n, dtype=np.int32)
    for p in range(n):
        seg = tokens[p:p + max_span]
        spans[p, :seg.shape[0]] = seg
        lens[p] = seg.shape[0]
    return spans, lens
