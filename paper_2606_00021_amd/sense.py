"""Python binding of ``libsense.so`` (the SENSE hot-path C ABI, include/sense.h).

Argument marshalling only: every step of retrieval and verification runs in
the library's HIP kernels.  PyTorch provides device memory (the tensors passed
in, the outputs and workspaces allocated here) and the current HIP stream.
There is no CPU fallback: if the library is missing or the tensors are not on
a GPU, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

# SENSE_LIB names another build of the same library to load instead (the
# test-suite's host-sanitizer build); by default the in-tree libsense.so.
LIB_PATH = os.environ.get("SENSE_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libsense.so")

SENSE_OK = 0
STATUS_NAMES = {
    0: "SENSE_OK",
    1: "SENSE_ERR_INVALID_ARGUMENT",
    2: "SENSE_ERR_MISALIGNED",
    3: "SENSE_ERR_UNSUPPORTED",
    4: "SENSE_ERR_OUT_OF_MEMORY",
    5: "SENSE_ERR_WORKSPACE",
    6: "SENSE_ERR_HIP",
}
SENSE_F32, SENSE_F16, SENSE_BF16 = 0, 1, 2
METRICS = {"ip": 0, "cosine": 1}
SENSE_INDEX_COPY_KEYS = 1

_TORCH_DTYPE = {torch.float32: SENSE_F32, torch.float16: SENSE_F16, torch.bfloat16: SENSE_BF16}

# Every symbol include/sense.h declares.
EXPORTED = (
    "sense_build_index",
    "sense_destroy_index",
    "sense_index_info",
    "sense_retrieve_workspace_size",
    "sense_retrieve",
    "sense_retrieve_noalloc",
    "sense_retrieve_noalloc_max_bytes",
    "sense_soft_gate_verify_workspace_size",
    "sense_soft_gate_verify",
    "sense_build_dynamic_index",
    "sense_index_append",
    "sense_select_candidates",
    "sense_build_loose_trie",
    "sense_soft_gate_verify_tree_workspace_size",
    "sense_soft_gate_verify_tree",
    "sense_project_workspace_size",
    "sense_project",
    "sense_ivf_assign",
    "sense_pq_encode",
    "sense_build_ivf_index",
    "sense_ivf_search_workspace_size",
    "sense_ivf_search",
    "sense_set_timer_events",
    "sense_read_bandwidth_probe",
    "sense_status_string",
    "sense_last_error_message",
)
SENSE_TIMER_SCAN, SENSE_TIMER_TOPK, SENSE_TIMER_VERIFY, SENSE_TIMER_SELECT = 0, 1, 2, 3
SENSE_TIMER_TRIE, SENSE_TIMER_PROJECT, SENSE_TIMER_IVF, SENSE_TIMER_FILTER = 4, 5, 6, 7


class SenseError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        self.status_name = STATUS_NAMES.get(status, str(status))
        super().__init__(f"{where}: {self.status_name}: {detail}")


class IndexDesc(ctypes.Structure):
    _fields_ = [
        ("keys", ctypes.c_void_p),
        ("key_dtype", ctypes.c_int),
        ("n", ctypes.c_int64),
        ("d", ctypes.c_int32),
        ("key_stride", ctypes.c_int64),
        ("spans", ctypes.c_void_p),
        ("max_span", ctypes.c_int32),
        ("span_len", ctypes.c_void_p),
        ("metric", ctypes.c_int),
        ("flags", ctypes.c_uint32),
    ]


class DynamicIndexDesc(ctypes.Structure):
    _fields_ = [
        ("key_dtype", ctypes.c_int),
        ("d", ctypes.c_int32),
        ("capacity", ctypes.c_int64),
        ("max_span", ctypes.c_int32),
        ("metric", ctypes.c_int),
    ]


class SelectParams(ctypes.Structure):
    _fields_ = [
        ("alpha", ctypes.c_float),
        ("beta", ctypes.c_float),
        ("delta", ctypes.c_float),
        ("anchor_override", ctypes.c_int32),
    ]


class TrieDesc(ctypes.Structure):
    _fields_ = [
        ("order", ctypes.c_void_p),
        ("gamma", ctypes.c_void_p),
        ("tree_tokens", ctypes.c_void_p),
        ("tree_parent", ctypes.c_void_p),
        ("tree_depth", ctypes.c_void_p),
        ("tree_cand", ctypes.c_void_p),
        ("tree_len", ctypes.c_void_p),
        ("sorted_drafts", ctypes.c_void_p),
        ("sorted_len", ctypes.c_void_p),
        ("mask", ctypes.c_void_p),
        ("mask_ld", ctypes.c_int64),
        ("full_mask", ctypes.c_void_p),
        ("full_mask_dtype", ctypes.c_int),
        ("prefix_len", ctypes.c_int32),
        ("cache_len", ctypes.c_int64),
    ]


class ProjDesc(ctypes.Structure):
    _fields_ = [
        ("mean", ctypes.c_void_p),
        ("basis", ctypes.c_void_p),
        ("d_in", ctypes.c_int32),
        ("d_out", ctypes.c_int32),
        ("normalize", ctypes.c_int32),
    ]


class IvfDesc(ctypes.Structure):
    _fields_ = [
        ("keys", ctypes.c_void_p),
        ("key_dtype", ctypes.c_int),
        ("n", ctypes.c_int64),
        ("d", ctypes.c_int32),
        ("key_stride", ctypes.c_int64),
        ("spans", ctypes.c_void_p),
        ("max_span", ctypes.c_int32),
        ("span_len", ctypes.c_void_p),
        ("metric", ctypes.c_int),
        ("centroids", ctypes.c_void_p),
        ("nlist", ctypes.c_int32),
        ("list_ids", ctypes.c_void_p),
        ("pq_codebooks", ctypes.c_void_p),
        ("pq_m", ctypes.c_int32),
        ("pq_ksub", ctypes.c_int32),
        ("pq_codes", ctypes.c_void_p),
    ]


class GateParams(ctypes.Structure):
    _fields_ = [
        ("gamma", ctypes.c_float),
        ("topk", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("tau", ctypes.c_int32),
        ("entropy_normalized", ctypes.c_int32),
    ]


_lib = None


def load_library() -> ctypes.CDLL:
    """Load libsense.so and declare its signatures (no device work)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run paper_2606_00021_amd.build.build() "
            "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    PP = ctypes.POINTER(ctypes.c_void_p)
    PSZ = ctypes.POINTER(ctypes.c_size_t)
    sig = {
        "sense_build_index": [ctypes.POINTER(IndexDesc), P, PP],
        "sense_destroy_index": [P],
        "sense_index_info": [P, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int32),
                             ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int),
                             ctypes.POINTER(ctypes.c_int)],
        "sense_retrieve_workspace_size": [P, I32, I32, PSZ],
        "sense_retrieve": [P, P, ctypes.c_int, I32, I32, P, P, P, P, P, SZ, P],
        "sense_retrieve_noalloc": [P, P, ctypes.c_int, I32, I32, P, P, P, P, P],
        "sense_soft_gate_verify_workspace_size": [I32, I32, I32, PSZ],
        "sense_build_dynamic_index": [ctypes.POINTER(DynamicIndexDesc), PP],
        "sense_index_append": [P, P, ctypes.c_int, P, I32, P],
        "sense_select_candidates": [P, P, P, I32, P, P, P, I32, P, I32, I32, I32,
                                    ctypes.POINTER(SelectParams), P, P, P, P, P],
        "sense_soft_gate_verify": [P, ctypes.c_int, I64, P, P, I32, I32, I32, I32,
                                   ctypes.POINTER(GateParams), P, P, P, P, P, P, SZ, P],
        "sense_build_loose_trie": [P, P, I32, I32, I32, ctypes.POINTER(TrieDesc), P],
        "sense_project_workspace_size": [ctypes.POINTER(ProjDesc), ctypes.c_int, I64, PSZ],
        "sense_ivf_assign": [P, ctypes.c_int, I64, I32, I64, P, I32, ctypes.c_int, P, P],
        "sense_pq_encode": [P, ctypes.c_int, I64, I32, I64, P, I32, P, P, I32, I32, P, P],
        "sense_build_ivf_index": [ctypes.POINTER(IvfDesc), P, PP],
        "sense_ivf_search_workspace_size": [P, I32, I32, I32, PSZ],
        "sense_ivf_search": [P, P, ctypes.c_int, I32, I32, I32, P, P, P, P, P, P, SZ, P],
        "sense_project": [ctypes.POINTER(ProjDesc), P, ctypes.c_int, I64, I64, P, ctypes.c_int,
                          I64, P, SZ, P],
        "sense_soft_gate_verify_tree_workspace_size": [I32, I32, I32, I32, PSZ],
        "sense_soft_gate_verify_tree": [P, ctypes.c_int, I64, P, P, P, P, I32, I32, I32, I32,
                                        ctypes.POINTER(GateParams), P, P, P, P, P, P, SZ, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.sense_read_bandwidth_probe.argtypes = [P, SZ, P, P]
    lib.sense_read_bandwidth_probe.restype = ctypes.c_int
    lib.sense_set_timer_events.argtypes = [ctypes.c_int, P, P]
    lib.sense_set_timer_events.restype = ctypes.c_int
    lib.sense_status_string.argtypes = [ctypes.c_int]
    lib.sense_status_string.restype = ctypes.c_char_p
    lib.sense_last_error_message.argtypes = []
    lib.sense_last_error_message.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int, where: str) -> None:
    if status != SENSE_OK:
        detail = load_library().sense_last_error_message().decode(errors="replace")
        raise SenseError(status, where, detail)


def _dev_ptr(t: torch.Tensor | None, name: str):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    return ctypes.c_void_p(t.data_ptr())


def _stream_handle(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


@dataclass
class Index:
    """A built datastore index.  Holds references to the borrowed tensors so
    they outlive the handle."""

    handle: ctypes.c_void_p
    keys: torch.Tensor
    spans: torch.Tensor
    span_len: torch.Tensor | None
    n: int
    d: int
    max_span: int
    metric: str

    def close(self) -> None:
        if self.handle:
            h, self.handle = self.handle, None
            _check(load_library().sense_destroy_index(h), "sense_destroy_index")

    def __del__(self):  # best effort; explicit close() reports errors
        try:
            self.close()
        except Exception:
            pass


def sense_build_index(keys: torch.Tensor, spans: torch.Tensor, span_len: torch.Tensor | None = None,
                      metric: str = "cosine", copy_keys: bool = False, stream=None) -> Index:
    """Build the datastore index over ``keys`` (N x d fp16/bf16, rows may be
    strided) with continuations ``spans`` (N x M int32) and optional
    ``span_len`` (N int32)."""
    lib = load_library()
    if keys.dim() != 2 or keys.dtype not in (torch.float16, torch.bfloat16):
        raise ValueError("keys must be a 2-D float16/bfloat16 tensor")
    if keys.stride(1) != 1:
        raise ValueError("keys rows must be contiguous (stride(1) == 1)")
    if spans.dtype != torch.int32 or spans.dim() != 2 or not spans.is_contiguous():
        raise ValueError("spans must be a contiguous N x M int32 tensor")
    if span_len is not None and (span_len.dtype != torch.int32 or not span_len.is_contiguous()):
        raise ValueError("span_len must be a contiguous int32 tensor")
    desc = IndexDesc(
        keys=_dev_ptr(keys, "keys"), key_dtype=_TORCH_DTYPE[keys.dtype], n=keys.shape[0],
        d=keys.shape[1], key_stride=keys.stride(0), spans=_dev_ptr(spans, "spans"),
        max_span=spans.shape[1], span_len=_dev_ptr(span_len, "span_len"),
        metric=METRICS[metric], flags=SENSE_INDEX_COPY_KEYS if copy_keys else 0)
    handle = ctypes.c_void_p()
    _check(lib.sense_build_index(ctypes.byref(desc), _stream_handle(stream), ctypes.byref(handle)),
           "sense_build_index")
    return Index(handle, keys, spans, span_len, keys.shape[0], keys.shape[1], spans.shape[1], metric)


class DynamicIndex:
    """A dynamic context cache (owned device memory; grows by append)."""

    def __init__(self, handle: ctypes.c_void_p, d: int, capacity: int, max_span: int,
                 metric: str, key_dtype: torch.dtype):
        self.handle = handle
        self.d = d
        self.capacity = capacity
        self.max_span = max_span
        self.metric = metric
        self.key_dtype = key_dtype

    @property
    def n(self) -> int:
        n = ctypes.c_int64()
        _check(load_library().sense_index_info(self.handle, ctypes.byref(n), None, None, None,
                                               None), "sense_index_info")
        return n.value

    def close(self) -> None:
        if self.handle:
            h, self.handle = self.handle, None
            _check(load_library().sense_destroy_index(h), "sense_destroy_index")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def sense_build_dynamic_index(d: int, capacity: int, max_span: int,
                              key_dtype: torch.dtype = torch.bfloat16,
                              metric: str = "cosine") -> DynamicIndex:
    """Create an empty dynamic context cache of ``capacity`` rows."""
    lib = load_library()
    if key_dtype not in (torch.float16, torch.bfloat16):
        raise ValueError("key_dtype must be float16 or bfloat16")
    desc = DynamicIndexDesc(key_dtype=_TORCH_DTYPE[key_dtype], d=d, capacity=capacity,
                            max_span=max_span, metric=METRICS[metric])
    handle = ctypes.c_void_p()
    _check(lib.sense_build_dynamic_index(ctypes.byref(desc), ctypes.byref(handle)),
           "sense_build_dynamic_index")
    return DynamicIndex(handle, d, capacity, max_span, metric, key_dtype)


def sense_index_append(index: DynamicIndex, keys: torch.Tensor, tokens: torch.Tensor,
                       stream=None) -> None:
    """Append generated positions: ``keys`` (count x d, fp32/fp16/bf16,
    contiguous; row j predicted tokens[j]) and ``tokens`` (count int32)."""
    if keys.dim() == 1:
        keys = keys.unsqueeze(0)
    if keys.dtype not in _TORCH_DTYPE or not keys.is_contiguous() or keys.shape[1] != index.d:
        raise ValueError("keys must be a contiguous count x d float32/float16/bfloat16 tensor")
    if tokens.dtype != torch.int32 or not tokens.is_contiguous() or tokens.numel() != keys.shape[0]:
        raise ValueError("tokens must be a contiguous int32 tensor with one id per key row")
    _check(load_library().sense_index_append(index.handle, _dev_ptr(keys, "keys"),
                                             _TORCH_DTYPE[keys.dtype], _dev_ptr(tokens, "tokens"),
                                             keys.shape[0], _stream_handle(stream)),
           "sense_index_append")


def sense_select_candidates(static: tuple, dynamic: tuple | None, anchors: torch.Tensor,
                            top_n: int, alpha: float, beta: float, delta: float = 0.0,
                            anchor_override: bool = True, out: tuple | None = None,
                            stream=None):
    """Composite-score Top-N over each query's static and dynamic hits.

    ``static`` and ``dynamic`` are (scores [Q,n] fp32, drafts [Q,n,M] int32,
    lengths [Q,n] int32 or None) as sense_retrieve returns them (``dynamic``
    may be None).  Returns (drafts [Q,top_n,M], lengths [Q,top_n], source
    [Q,top_n] positions in the pool, composite scores [Q,top_n])."""
    lib = load_library()

    def parts(t):
        if t is None:
            return None, None, None, 0
        sc, dr, ln = t
        for x, nm in ((sc, "scores"), (dr, "drafts"), (ln, "lengths")):
            if x is not None and not x.is_contiguous():
                raise ValueError(f"{nm} must be contiguous")
        if sc.dtype != torch.float32 or dr.dtype != torch.int32 or dr.dim() != 3:
            raise ValueError("scores must be fp32 [Q,n] and drafts int32 [Q,n,M]")
        if ln is not None and ln.dtype != torch.int32:
            raise ValueError("lengths must be int32")
        return sc, dr, ln, sc.shape[-1]

    ss, ds, ls, ns = parts(static)
    sd, dd, ld, nd = parts(dynamic)
    ref = ds if ds is not None else dd
    nq, m = ref.shape[0], ref.shape[2]
    if anchors.dtype != torch.int32 or anchors.numel() != nq or not anchors.is_contiguous():
        raise ValueError("anchors must be a contiguous int32 tensor of one id per query")
    dev = anchors.device
    if out is None:
        out = (torch.empty((nq, top_n, m), dtype=torch.int32, device=dev),
               torch.empty((nq, top_n), dtype=torch.int32, device=dev),
               torch.empty((nq, top_n), dtype=torch.int32, device=dev),
               torch.empty((nq, top_n), dtype=torch.float32, device=dev))
    odr, oln, osrc, osc = out
    params = SelectParams(alpha=alpha, beta=beta, delta=delta,
                          anchor_override=int(bool(anchor_override)))
    _check(lib.sense_select_candidates(
        _dev_ptr(ss, "static_scores"), _dev_ptr(ds, "static_drafts"), _dev_ptr(ls, "static_len"),
        ns, _dev_ptr(sd, "dynamic_scores"), _dev_ptr(dd, "dynamic_drafts"),
        _dev_ptr(ld, "dynamic_len"), nd, _dev_ptr(anchors, "anchors"), nq, m, top_n,
        ctypes.byref(params), _dev_ptr(odr, "out_drafts"), _dev_ptr(oln, "out_len"),
        _dev_ptr(osrc, "out_source"), _dev_ptr(osc, "out_score"), _stream_handle(stream)),
        "sense_select_candidates")
    return out


def sense_retrieve_workspace_size(index: Index, n_queries: int, k: int) -> int:
    size = ctypes.c_size_t()
    _check(load_library().sense_retrieve_workspace_size(index.handle, n_queries, k,
                                                        ctypes.byref(size)),
           "sense_retrieve_workspace_size")
    return size.value


def sense_retrieve(index: Index, queries: torch.Tensor, k: int, workspace: torch.Tensor | None = None,
                   out: tuple | None = None, stream=None):
    """Exact top-k retrieval for ``queries`` (Q x d, fp32 or the key dtype).

    Returns (ids int64 [Q,k], scores fp32 [Q,k], drafts int32 [Q,k,M],
    draft_len int32 [Q,k]).  ``out`` may supply those four tensors and
    ``workspace`` a uint8 tensor of sense_retrieve_workspace_size bytes."""
    lib = load_library()
    if queries.dim() == 1:
        queries = queries.unsqueeze(0)
    if queries.dtype not in _TORCH_DTYPE or not queries.is_contiguous():
        raise ValueError("queries must be a contiguous float32/float16/bfloat16 tensor")
    if queries.shape[1] != index.d:
        raise ValueError(f"queries have d={queries.shape[1]}, index has d={index.d}")
    nq = queries.shape[0]
    dev = queries.device
    if out is None:
        ids = torch.empty((nq, k), dtype=torch.int64, device=dev)
        scores = torch.empty((nq, k), dtype=torch.float32, device=dev)
        drafts = torch.empty((nq, k, index.max_span), dtype=torch.int32, device=dev)
        dlen = torch.empty((nq, k), dtype=torch.int32, device=dev)
    else:
        ids, scores, drafts, dlen = out
    if workspace is None:
        workspace = torch.empty(max(sense_retrieve_workspace_size(index, nq, k), 1),
                                dtype=torch.uint8, device=dev)
    _check(lib.sense_retrieve(index.handle, _dev_ptr(queries, "queries"), _TORCH_DTYPE[queries.dtype],
                              nq, k, _dev_ptr(ids, "out_ids"), _dev_ptr(scores, "out_scores"),
                              _dev_ptr(drafts, "out_drafts"), _dev_ptr(dlen, "out_draft_len"),
                              _dev_ptr(workspace, "workspace"), workspace.numel(),
                              _stream_handle(stream)),
           "sense_retrieve")
    return ids, scores, drafts, dlen


def sense_retrieve_noalloc_max_bytes() -> int:
    """Bytes of the library's static scratch that sense_retrieve_noalloc uses."""
    lib = load_library()
    lib.sense_retrieve_noalloc_max_bytes.restype = ctypes.c_size_t
    lib.sense_retrieve_noalloc_max_bytes.argtypes = []
    return int(lib.sense_retrieve_noalloc_max_bytes())


def sense_retrieve_noalloc(index: Index, queries: torch.Tensor, k: int, out: tuple,
                           stream=None):
    """sense_retrieve with the library's static scratch instead of a
    workspace: allocates nothing, so ``out`` (ids, scores, drafts, draft_len)
    is required.  Calls overlapping on one device race on that scratch."""
    lib = load_library()
    if queries.dim() == 1:
        queries = queries.unsqueeze(0)
    if queries.dtype not in _TORCH_DTYPE or not queries.is_contiguous():
        raise ValueError("queries must be a contiguous float32/float16/bfloat16 tensor")
    if queries.shape[1] != index.d:
        raise ValueError(f"queries have d={queries.shape[1]}, index has d={index.d}")
    ids, scores, drafts, dlen = out
    _check(lib.sense_retrieve_noalloc(index.handle, _dev_ptr(queries, "queries"),
                                      _TORCH_DTYPE[queries.dtype], queries.shape[0], k,
                                      _dev_ptr(ids, "out_ids"), _dev_ptr(scores, "out_scores"),
                                      _dev_ptr(drafts, "out_drafts"),
                                      _dev_ptr(dlen, "out_draft_len"), _stream_handle(stream)),
           "sense_retrieve_noalloc")
    return ids, scores, drafts, dlen


def sense_soft_gate_verify_workspace_size(n_cand: int, max_len: int, vocab: int) -> int:
    size = ctypes.c_size_t()
    _check(load_library().sense_soft_gate_verify_workspace_size(n_cand, max_len, vocab,
                                                                ctypes.byref(size)),
           "sense_soft_gate_verify_workspace_size")
    return size.value


def sense_soft_gate_verify(logits: torch.Tensor, drafts: torch.Tensor,
                           draft_len: torch.Tensor | None = None, n_groups: int = 1,
                           gamma: float = 0.05, topk: int = 3, window: int = 6, tau: int = 0,
                           entropy_normalized: bool = True, vocab: int | None = None,
                           want_gate_score: bool = True, want_masks: bool = True,
                           want_rank: bool = True, workspace: torch.Tensor | None = None,
                           out: dict | None = None, stream=None) -> dict:
    """Soft-gated evaluation of drafts (C x M int32) against aligned logits
    (C x M x stride, rows contiguous).  Returns a dict of device tensors:
    accept_len [C], best [n_groups], and optionally gate_score [C,M] fp32,
    masks [C,M] uint8, rank [C,M] int32."""
    lib = load_library()
    if drafts.dtype != torch.int32 or drafts.dim() != 2 or not drafts.is_contiguous():
        raise ValueError("drafts must be a contiguous C x M int32 tensor")
    c, m = drafts.shape
    if logits.dtype not in _TORCH_DTYPE or logits.dim() != 3 or tuple(logits.shape[:2]) != (c, m):
        raise ValueError("logits must be C x M x V float32/float16/bfloat16")
    if logits.stride(2) != 1:
        raise ValueError("logits rows must be contiguous (stride(2) == 1)")
    row_stride = logits.stride(1) if m > 1 else logits.stride(0)
    if m > 1 and logits.stride(0) != m * row_stride:
        raise ValueError("logits must have stride(0) == M * stride(1)")
    if draft_len is not None and (draft_len.dtype != torch.int32 or not draft_len.is_contiguous()
                                  or draft_len.numel() != c):
        raise ValueError("draft_len must be a contiguous int32 tensor of C entries")
    v = logits.shape[2] if vocab is None else vocab
    dev = drafts.device
    if out is None:
        out = {"accept_len": torch.empty(c, dtype=torch.int32, device=dev),
               "best": torch.empty(max(n_groups, 1), dtype=torch.int32, device=dev)}
        if want_gate_score:
            out["gate_score"] = torch.empty((c, m), dtype=torch.float32, device=dev)
        if want_masks:
            out["masks"] = torch.empty((c, m), dtype=torch.uint8, device=dev)
        if want_rank:
            out["rank"] = torch.empty((c, m), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(sense_soft_gate_verify_workspace_size(c, m, v), 1),
                                dtype=torch.uint8, device=dev)
    params = GateParams(gamma=gamma, topk=topk, window=window, tau=tau,
                        entropy_normalized=int(bool(entropy_normalized)))
    _check(lib.sense_soft_gate_verify(
        _dev_ptr(logits, "logits"), _TORCH_DTYPE[logits.dtype], row_stride,
        _dev_ptr(drafts, "drafts"), _dev_ptr(draft_len, "draft_len"), c, m, v, n_groups,
        ctypes.byref(params), _dev_ptr(out["accept_len"], "out_accept_len"),
        _dev_ptr(out["best"], "out_best"), _dev_ptr(out.get("gate_score"), "out_gate_score"),
        _dev_ptr(out.get("masks"), "out_masks"), _dev_ptr(out.get("rank"), "out_rank"),
        _dev_ptr(workspace, "workspace"), workspace.numel(), _stream_handle(stream)),
        "sense_soft_gate_verify")
    return out


def sense_set_timer_events(which: int, start: "torch.cuda.Event | None",
                           stop: "torch.cuda.Event | None") -> None:
    """Have the next calls on this thread record ``start``/``stop`` around the
    kernels named by ``which`` (SENSE_TIMER_*); None switches it off."""
    sp = None if start is None else ctypes.c_void_p(start.cuda_event)
    ep = None if stop is None else ctypes.c_void_p(stop.cuda_event)
    if start is not None and (not sp.value or not ep.value):
        raise ValueError("record the events once before registering them (torch creates "
                         "the underlying hipEvent_t at the first record())")
    _check(load_library().sense_set_timer_events(which, sp, ep), "sense_set_timer_events")


def sense_read_bandwidth_probe(buf: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """Enqueue one plain streaming read of ``buf`` (a contiguous GPU tensor);
    ``sink`` is a 1-element int32/uint32 GPU tensor the kernel may write."""
    if not buf.is_contiguous():
        raise ValueError("buf must be contiguous")
    nbytes = buf.numel() * buf.element_size() // 16 * 16
    _check(load_library().sense_read_bandwidth_probe(_dev_ptr(buf, "buf"), nbytes,
                                                     _dev_ptr(sink, "sink"), _stream_handle(stream)),
           "sense_read_bandwidth_probe")


def sense_build_loose_trie(drafts: torch.Tensor, draft_len: torch.Tensor | None = None,
                           n_groups: int = 1, want_sorted: bool = True, want_mask: bool = False,
                           full_mask: dict | None = None, out: dict | None = None,
                           stream=None) -> dict:
    """LexSort + loose trie of each group of ``drafts`` (C x M int32).

    Returns a dict of device tensors: order [C], gamma [C,M] (sorted order),
    tree_tokens / tree_parent / tree_depth / tree_cand [G, nodes],
    tree_len [G], and optionally sorted_drafts [C,M], sorted_len [C],
    mask [G, nodes, nodes] uint8 and full_mask [G, nodes, cache_len]
    (``full_mask`` = {"dtype": torch dtype, "prefix_len": m, "cache_len": n})."""
    lib = load_library()
    if drafts.dtype != torch.int32 or drafts.dim() != 2 or not drafts.is_contiguous():
        raise ValueError("drafts must be a contiguous C x M int32 tensor")
    if draft_len is not None and (draft_len.dtype != torch.int32 or not draft_len.is_contiguous()
                                  or draft_len.numel() != drafts.shape[0]):
        raise ValueError("draft_len must be a contiguous int32 tensor of C entries")
    c, m = drafts.shape
    if n_groups < 1 or c % n_groups:
        raise ValueError("n_groups must divide the number of drafts")
    nodes = c // n_groups * m
    dev = drafts.device
    if out is None:
        i32 = dict(dtype=torch.int32, device=dev)
        out = {"order": torch.empty(c, **i32), "gamma": torch.empty((c, m), **i32),
               "tree_tokens": torch.empty((n_groups, nodes), **i32),
               "tree_parent": torch.empty((n_groups, nodes), **i32),
               "tree_depth": torch.empty((n_groups, nodes), **i32),
               "tree_cand": torch.empty((n_groups, nodes), **i32),
               "tree_len": torch.empty(n_groups, **i32)}
        if want_sorted:
            out["sorted_drafts"] = torch.empty((c, m), **i32)
            out["sorted_len"] = torch.empty(c, **i32)
        if want_mask:
            out["mask"] = torch.zeros((n_groups, nodes, nodes), dtype=torch.uint8, device=dev)
        if full_mask is not None:
            out["full_mask"] = torch.zeros((n_groups, nodes, full_mask["cache_len"]),
                                           dtype=full_mask["dtype"], device=dev)
    fm = out.get("full_mask")
    if fm is not None and full_mask is None:
        raise ValueError("out holds a full_mask: pass full_mask={'prefix_len': ...} as well")
    desc = TrieDesc(
        order=_dev_ptr(out["order"], "order"), gamma=_dev_ptr(out["gamma"], "gamma"),
        tree_tokens=_dev_ptr(out["tree_tokens"], "tree_tokens"),
        tree_parent=_dev_ptr(out["tree_parent"], "tree_parent"),
        tree_depth=_dev_ptr(out["tree_depth"], "tree_depth"),
        tree_cand=_dev_ptr(out["tree_cand"], "tree_cand"),
        tree_len=_dev_ptr(out["tree_len"], "tree_len"),
        sorted_drafts=_dev_ptr(out.get("sorted_drafts"), "sorted_drafts"),
        sorted_len=_dev_ptr(out.get("sorted_len"), "sorted_len"),
        mask=_dev_ptr(out.get("mask"), "mask"),
        mask_ld=out["mask"].shape[-1] if "mask" in out else 0,
        full_mask=_dev_ptr(fm, "full_mask"),
        full_mask_dtype=_TORCH_DTYPE[fm.dtype] if fm is not None else 0,
        prefix_len=full_mask["prefix_len"] if full_mask is not None else 0,
        cache_len=fm.shape[-1] if fm is not None else 0)
    _check(lib.sense_build_loose_trie(_dev_ptr(drafts, "drafts"), _dev_ptr(draft_len, "draft_len"),
                                      c, m, n_groups, ctypes.byref(desc), _stream_handle(stream)),
           "sense_build_loose_trie")
    return out


def sense_soft_gate_verify_tree_workspace_size(n_cand: int, max_len: int, vocab: int,
                                               n_groups: int) -> int:
    size = ctypes.c_size_t()
    _check(load_library().sense_soft_gate_verify_tree_workspace_size(
        n_cand, max_len, vocab, n_groups, ctypes.byref(size)),
        "sense_soft_gate_verify_tree_workspace_size")
    return size.value


def sense_soft_gate_verify_tree(logits: torch.Tensor, trie: dict, n_groups: int = 1,
                                gamma: float = 0.05, topk: int = 3, window: int = 6,
                                tau: int = 0, entropy_normalized: bool = True,
                                vocab: int | None = None, want_gate_score: bool = True,
                                want_masks: bool = True, want_rank: bool = True,
                                workspace: torch.Tensor | None = None, out: dict | None = None,
                                stream=None) -> dict:
    """Soft-gated evaluation through the loose trie.  ``logits`` holds per
    group 1 + nodes rows (G x (1 + nodes) x V, or (G * (1 + nodes)) x V):
    row 0 the current position's distribution, row 1 + u the distribution
    after tree node u.  ``trie`` is sense_build_loose_trie's result.  Returns
    the outputs of sense_soft_gate_verify, per draft in sorted order."""
    lib = load_library()
    gam = trie["gamma"]
    c, m = gam.shape
    if logits.dtype not in _TORCH_DTYPE or logits.stride(-1) != 1:
        raise ValueError("logits must be float32/float16/bfloat16 with contiguous rows")
    rows = logits.reshape(-1, logits.shape[-1]) if logits.dim() == 3 else logits
    if rows.dim() != 2 or rows.shape[0] != n_groups * (1 + c // n_groups * m):
        raise ValueError("logits must hold n_groups x (1 + nodes) rows")
    row_stride = rows.stride(0)
    v = rows.shape[1] if vocab is None else vocab
    dev = gam.device
    if out is None:
        out = {"accept_len": torch.empty(c, dtype=torch.int32, device=dev),
               "best": torch.empty(max(n_groups, 1), dtype=torch.int32, device=dev)}
        if want_gate_score:
            out["gate_score"] = torch.empty((c, m), dtype=torch.float32, device=dev)
        if want_masks:
            out["masks"] = torch.empty((c, m), dtype=torch.uint8, device=dev)
        if want_rank:
            out["rank"] = torch.empty((c, m), dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(sense_soft_gate_verify_tree_workspace_size(c, m, v, n_groups),
                                    1), dtype=torch.uint8, device=dev)
    params = GateParams(gamma=gamma, topk=topk, window=window, tau=tau,
                        entropy_normalized=int(bool(entropy_normalized)))
    _check(lib.sense_soft_gate_verify_tree(
        _dev_ptr(rows, "logits"), _TORCH_DTYPE[logits.dtype], row_stride,
        _dev_ptr(trie["tree_tokens"], "tree_tokens"), _dev_ptr(trie["tree_parent"], "tree_parent"),
        _dev_ptr(trie["tree_len"], "tree_len"), _dev_ptr(gam, "gamma"), c, m, v, n_groups,
        ctypes.byref(params), _dev_ptr(out["accept_len"], "out_accept_len"),
        _dev_ptr(out["best"], "out_best"), _dev_ptr(out.get("gate_score"), "out_gate_score"),
        _dev_ptr(out.get("masks"), "out_masks"), _dev_ptr(out.get("rank"), "out_rank"),
        _dev_ptr(workspace, "workspace"), workspace.numel(), _stream_handle(stream)),
        "sense_soft_gate_verify_tree")
    return out


def _proj_desc(basis: torch.Tensor, mean: torch.Tensor | None, normalize: bool) -> ProjDesc:
    if basis.dtype != torch.float32 or basis.dim() != 2 or not basis.is_contiguous():
        raise ValueError("basis must be a contiguous d_out x d_in float32 tensor")
    if mean is not None and (mean.dtype != torch.float32 or not mean.is_contiguous()
                             or mean.numel() != basis.shape[1]):
        raise ValueError("mean must be a contiguous float32 tensor of d_in entries")
    return ProjDesc(mean=_dev_ptr(mean, "mean"), basis=_dev_ptr(basis, "basis"),
                    d_in=basis.shape[1], d_out=basis.shape[0], normalize=int(bool(normalize)))


def sense_project_workspace_size(basis: torch.Tensor, x_dtype: torch.dtype, n_rows: int,
                                 mean: torch.Tensor | None = None, normalize: bool = True) -> int:
    size = ctypes.c_size_t()
    desc = _proj_desc(basis, mean, normalize)
    _check(load_library().sense_project_workspace_size(ctypes.byref(desc), _TORCH_DTYPE[x_dtype],
                                                       n_rows, ctypes.byref(size)),
           "sense_project_workspace_size")
    return size.value


def sense_project(x: torch.Tensor, basis: torch.Tensor, mean: torch.Tensor | None = None,
                  normalize: bool = True, out_dtype: torch.dtype = torch.float32,
                  out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                  stream=None) -> torch.Tensor:
    """PCA projection (+ L2 normalisation) of the rows of ``x`` (n x d_in,
    rows may be strided) with ``basis`` (d_out x d_in fp32, principal
    directions as rows) and ``mean`` (d_in fp32 or None).  Returns n x d_out
    of ``out_dtype`` (or writes ``out``)."""
    if x.dim() == 1:
        x = x.unsqueeze(0)
    if x.dtype not in _TORCH_DTYPE or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D float32/float16/bfloat16 tensor with contiguous rows")
    desc = _proj_desc(basis, mean, normalize)
    n = x.shape[0]
    if x.shape[1] != desc.d_in:
        raise ValueError(f"x has {x.shape[1]} columns, basis expects {desc.d_in}")
    if out is None:
        out = torch.empty((n, desc.d_out), dtype=out_dtype, device=x.device)
    if out.dim() != 2 or out.stride(1) != 1 or out.shape[0] != n:
        raise ValueError("out must be n x (>= d_out) with contiguous rows")
    if workspace is None:
        need = sense_project_workspace_size(basis, x.dtype, n, mean, normalize)
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    _check(load_library().sense_project(
        ctypes.byref(desc), _dev_ptr(x, "x"), _TORCH_DTYPE[x.dtype], n, x.stride(0),
        _dev_ptr(out, "out"), _TORCH_DTYPE[out.dtype], out.stride(0), _dev_ptr(workspace, "workspace"),
        workspace.numel(), _stream_handle(stream)), "sense_project")
    return out


def _keys_2d(keys: torch.Tensor):
    if keys.dim() != 2 or keys.dtype not in (torch.float16, torch.bfloat16) or keys.stride(1) != 1:
        raise ValueError("keys must be a 2-D float16/bfloat16 tensor with contiguous rows")
    return keys.shape[0], keys.shape[1], keys.stride(0)


def sense_ivf_assign(keys: torch.Tensor, centroids: torch.Tensor, metric: str = "cosine",
                     out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Most similar centroid of every key row (int32 [n])."""
    n, d, ld = _keys_2d(keys)
    if centroids.dtype != torch.float32 or not centroids.is_contiguous() or centroids.shape[1] != d:
        raise ValueError("centroids must be a contiguous nlist x d float32 tensor")
    if out is None:
        out = torch.empty(n, dtype=torch.int32, device=keys.device)
    _check(load_library().sense_ivf_assign(_dev_ptr(keys, "keys"), _TORCH_DTYPE[keys.dtype], n, d,
                                           ld, _dev_ptr(centroids, "centroids"), centroids.shape[0],
                                           METRICS[metric], _dev_ptr(out, "out_list"),
                                           _stream_handle(stream)), "sense_ivf_assign")
    return out


def sense_pq_encode(keys: torch.Tensor, centroids: torch.Tensor, list_ids: torch.Tensor,
                    codebooks: torch.Tensor, out: torch.Tensor | None = None,
                    stream=None) -> torch.Tensor:
    """PQ codes (uint8 [n, m]) of the residuals key - centroid[list];
    codebooks is m x ksub x (d/m) float32."""
    n, d, ld = _keys_2d(keys)
    if codebooks.dtype != torch.float32 or codebooks.dim() != 3 or not codebooks.is_contiguous():
        raise ValueError("codebooks must be a contiguous m x ksub x dsub float32 tensor")
    m, ksub, _ = codebooks.shape
    if out is None:
        out = torch.empty((n, m), dtype=torch.uint8, device=keys.device)
    _check(load_library().sense_pq_encode(
        _dev_ptr(keys, "keys"), _TORCH_DTYPE[keys.dtype], n, d, ld, _dev_ptr(centroids, "centroids"),
        centroids.shape[0], _dev_ptr(list_ids, "list_ids"), _dev_ptr(codebooks, "codebooks"), m,
        ksub, _dev_ptr(out, "out_codes"), _stream_handle(stream)), "sense_pq_encode")
    return out


class IvfIndex:
    """An inverted-file index (owns its device memory; borrows the spans)."""

    def __init__(self, handle, d, nlist, max_span, metric, pq_m, spans, span_len):
        self.handle, self.d, self.nlist, self.max_span = handle, d, nlist, max_span
        self.metric, self.pq_m, self.spans, self.span_len = metric, pq_m, spans, span_len

    def close(self) -> None:
        if self.handle:
            h, self.handle = self.handle, None
            _check(load_library().sense_destroy_index(h), "sense_destroy_index")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def sense_build_ivf_index(keys: torch.Tensor | None, spans: torch.Tensor, centroids: torch.Tensor,
                          list_ids: torch.Tensor, span_len: torch.Tensor | None = None,
                          metric: str = "cosine", codebooks: torch.Tensor | None = None,
                          codes: torch.Tensor | None = None, key_dtype: torch.dtype | None = None,
                          stream=None) -> IvfIndex:
    """IVF-Flat (codebooks None) or IVF-PQ index.  For IVF-PQ ``keys`` may be
    None (then ``key_dtype`` names the query-compatible key type)."""
    lib = load_library()
    if keys is not None:
        n, d, ld = _keys_2d(keys)
        kdt = keys.dtype
    else:
        n, d, ld = list_ids.shape[0], centroids.shape[1], centroids.shape[1]
        kdt = key_dtype or torch.bfloat16
    m, ksub = (codebooks.shape[0], codebooks.shape[1]) if codebooks is not None else (0, 0)
    desc = IvfDesc(keys=_dev_ptr(keys, "keys"), key_dtype=_TORCH_DTYPE[kdt], n=n, d=d,
                   key_stride=ld, spans=_dev_ptr(spans, "spans"), max_span=spans.shape[1],
                   span_len=_dev_ptr(span_len, "span_len"), metric=METRICS[metric],
                   centroids=_dev_ptr(centroids, "centroids"), nlist=centroids.shape[0],
                   list_ids=_dev_ptr(list_ids, "list_ids"),
                   pq_codebooks=_dev_ptr(codebooks, "codebooks"), pq_m=m, pq_ksub=ksub,
                   pq_codes=_dev_ptr(codes, "codes"))
    handle = ctypes.c_void_p()
    _check(lib.sense_build_ivf_index(ctypes.byref(desc), _stream_handle(stream),
                                     ctypes.byref(handle)), "sense_build_ivf_index")
    return IvfIndex(handle, d, centroids.shape[0], spans.shape[1], metric, m, spans, span_len)


def sense_ivf_search_workspace_size(index: IvfIndex, n_queries: int, k: int, nprobe: int) -> int:
    size = ctypes.c_size_t()
    _check(load_library().sense_ivf_search_workspace_size(index.handle, n_queries, k, nprobe,
                                                          ctypes.byref(size)),
           "sense_ivf_search_workspace_size")
    return size.value


def sense_ivf_search(index: IvfIndex, queries: torch.Tensor, k: int, nprobe: int,
                     workspace: torch.Tensor | None = None, out: tuple | None = None,
                     want_probe: bool = False, stream=None):
    """Inverted-file search.  Returns (ids int64 [Q,k], scores fp32 [Q,k],
    drafts int32 [Q,k,M], draft_len int32 [Q,k]) and, with want_probe, the
    probed lists int64 [Q,nprobe]."""
    lib = load_library()
    if queries.dim() == 1:
        queries = queries.unsqueeze(0)
    if queries.dtype not in _TORCH_DTYPE or not queries.is_contiguous() or queries.shape[1] != index.d:
        raise ValueError("queries must be a contiguous Q x d float32/float16/bfloat16 tensor")
    nq = queries.shape[0]
    dev = queries.device
    if out is None:
        out = (torch.empty((nq, k), dtype=torch.int64, device=dev),
               torch.empty((nq, k), dtype=torch.float32, device=dev),
               torch.empty((nq, k, index.max_span), dtype=torch.int32, device=dev),
               torch.empty((nq, k), dtype=torch.int32, device=dev))
    probe = torch.empty((nq, nprobe), dtype=torch.int64, device=dev) if want_probe else None
    if workspace is None:
        workspace = torch.empty(max(sense_ivf_search_workspace_size(index, nq, k, nprobe), 1),
                                dtype=torch.uint8, device=dev)
    ids, sc, dr, dl = out
    _check(lib.sense_ivf_search(index.handle, _dev_ptr(queries, "queries"),
                                _TORCH_DTYPE[queries.dtype], nq, k, nprobe, _dev_ptr(ids, "ids"),
                                _dev_ptr(sc, "scores"), _dev_ptr(dr, "drafts"),
                                _dev_ptr(dl, "draft_len"), _dev_ptr(probe, "probe"),
                                _dev_ptr(workspace, "workspace"), workspace.numel(),
                                _stream_handle(stream)), "sense_ivf_search")
    return (ids, sc, dr, dl, probe) if want_probe else (ids, sc, dr, dl)
