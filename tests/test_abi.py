"""Host-side tests of the C ABI (no GPU needed, nothing is launched).

The library must load, export every entry point include/sense.h declares,
and reject bad arguments with the documented status before any device work.
Pointers passed here are fake, aligned addresses: each call returns during
validation, so none is dereferenced.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sense.h")

from paper_2606_00021_amd import sense  # noqa: E402

INVALID, MISALIGNED, UNSUPPORTED, WORKSPACE = 1, 2, 3, 5
FAKE = 1 << 20          # 1 MiB-aligned fake device address


@pytest.fixture(scope="module")
def lib():
    return sense.load_library()


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sense_[a-z_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_symbols() == sorted(sense.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_library_is_gfx950_only():
    # The embedded offload bundle names its target; only gfx950 is built.
    data = open(sense.LIB_PATH, "rb").read()
    assert b"gfx950" in data
    for other in (b"gfx942", b"gfx90a", b"gfx1100"):
        assert other not in data


def test_c_driver_refuses_bad_invocations_before_any_device_call():
    """The plain C caller (built with the library) prints its usage without an
    argument and rejects a directory without params.txt, both before its
    first HIP call, so this runs without a GPU."""
    import subprocess
    drv = os.path.join(ROOT, "tests", "c_abi", "sense_c_driver")
    assert os.access(drv, os.X_OK), "build the C driver first (__graft_entry__.build())"
    r = subprocess.run([drv], capture_output=True, text=True, timeout=60)
    assert r.returncode == 2 and "usage" in r.stderr
    r = subprocess.run([drv, os.path.join(ROOT, "tests", "c_abi", "no-such-dir")],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 1 and "params.txt" in r.stderr


def test_status_strings(lib):
    for code in range(7):
        assert lib.sense_status_string(code)
    assert lib.sense_status_string(99) == b"unknown status"


def p(x):
    return ctypes.c_void_p(x)


def desc(**kw):
    base = dict(keys=p(FAKE), key_dtype=sense.SENSE_BF16, n=1000, d=256, key_stride=256,
                spans=p(FAKE), max_span=8, span_len=None, metric=1, flags=0)
    base.update(kw)
    return sense.IndexDesc(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(keys=None), INVALID),
    (dict(spans=None), INVALID),
    (dict(key_dtype=sense.SENSE_F32), INVALID),
    (dict(n=0), INVALID),
    (dict(n=1 << 31), INVALID),
    (dict(d=0), INVALID),
    (dict(d=8200, key_stride=8200), INVALID),
    (dict(d=100, key_stride=104), INVALID),          # d % 8 != 0
    (dict(key_stride=128), INVALID),                 # stride < d
    (dict(max_span=0), INVALID),
    (dict(max_span=65), INVALID),
    (dict(metric=7), INVALID),
    (dict(flags=4), INVALID),
    (dict(keys=p(FAKE + 8)), MISALIGNED),
    (dict(key_stride=260), MISALIGNED),
])
def test_build_index_rejects(lib, kw, status):
    out = ctypes.c_void_p(123)
    d = desc(**kw)
    assert lib.sense_build_index(ctypes.byref(d), None, ctypes.byref(out)) == status
    assert out.value is None                         # *out cleared
    assert lib.sense_last_error_message()


def test_build_index_null_args(lib):
    out = ctypes.c_void_p()
    assert lib.sense_build_index(None, None, ctypes.byref(out)) == INVALID
    d = desc()
    assert lib.sense_build_index(ctypes.byref(d), None, None) == INVALID


def test_retrieve_rejects_null_index(lib):
    size = ctypes.c_size_t()
    assert lib.sense_retrieve_workspace_size(None, 1, 8, ctypes.byref(size)) == INVALID
    assert lib.sense_retrieve(None, p(FAKE), 0, 1, 8, p(FAKE), None, None, None, p(FAKE),
                              1 << 30, None) == INVALID
    assert lib.sense_destroy_index(None) == 0
    assert lib.sense_retrieve_noalloc(None, p(FAKE), 0, 1, 8, p(FAKE), None, None, None,
                                      None) == INVALID


def test_verify_row_limit_in_workspace_query(lib):
    size = ctypes.c_size_t()
    assert lib.sense_soft_gate_verify_workspace_size(1 << 18, 64, 1000,
                                                     ctypes.byref(size)) == UNSUPPORTED
    assert lib.sense_soft_gate_verify_workspace_size((1 << 18) - 1, 64, 1000,
                                                     ctypes.byref(size)) == 0


def test_noalloc_scratch_size(lib):
    lib.sense_retrieve_noalloc_max_bytes.restype = ctypes.c_size_t
    assert lib.sense_retrieve_noalloc_max_bytes() == 64 << 20


def verify_call(lib, **kw):
    a = dict(logits=p(FAKE), dtype=0, row_stride=1000, drafts=p(FAKE), draft_len=None,
             n_cand=8, max_len=8, vocab=1000, n_groups=1,
             params=sense.GateParams(gamma=0.05, topk=3, window=6, tau=0, entropy_normalized=1),
             acc=p(FAKE), best=p(FAKE), gs=None, masks=None, rank=None, ws=p(FAKE),
             ws_bytes=1 << 30)
    a.update(kw)
    prm = a["params"]
    return lib.sense_soft_gate_verify(
        a["logits"], a["dtype"], a["row_stride"], a["drafts"], a["draft_len"], a["n_cand"],
        a["max_len"], a["vocab"], a["n_groups"], None if prm is None else ctypes.byref(prm),
        a["acc"], a["best"], a["gs"], a["masks"], a["rank"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(params=None), INVALID),
    (dict(n_cand=-1), INVALID),
    (dict(max_len=0), INVALID),
    (dict(max_len=65), INVALID),
    (dict(vocab=0), INVALID),
    (dict(row_stride=999), INVALID),
    (dict(dtype=5), INVALID),
    (dict(n_groups=3), INVALID),                     # 8 % 3 != 0
    (dict(n_groups=0), INVALID),
    # 2^24 rows: one 256-thread block each would pass 2^32 work-items
    (dict(n_cand=1 << 18, max_len=64), UNSUPPORTED),
    (dict(n_cand=(1 << 24) + 3, max_len=1), UNSUPPORTED),
    (dict(logits=None), INVALID),
    (dict(drafts=None), INVALID),
    (dict(acc=None), INVALID),
    (dict(best=None), INVALID),
    (dict(params=sense.GateParams(gamma=0.05, topk=0, window=6, tau=0, entropy_normalized=1)), INVALID),
    (dict(params=sense.GateParams(gamma=0.05, topk=3, window=-1, tau=0, entropy_normalized=1)), INVALID),
    (dict(params=sense.GateParams(gamma=0.05, topk=3, window=65, tau=0, entropy_normalized=1)), INVALID),
    (dict(params=sense.GateParams(gamma=0.05, topk=3, window=6, tau=-1, entropy_normalized=1)), INVALID),
    (dict(params=sense.GateParams(gamma=float("nan"), topk=3, window=6, tau=0, entropy_normalized=1)), INVALID),
    (dict(ws=None), WORKSPACE),
    (dict(ws_bytes=16), WORKSPACE),
    (dict(ws=p(FAKE + 64)), MISALIGNED),
    (dict(logits=p(FAKE + 2)), MISALIGNED),          # fp32 logits off their element size
])
def test_verify_rejects(lib, kw, status):
    assert verify_call(lib, **kw) == status
    assert lib.sense_last_error_message()


def test_read_probe_rejects(lib):
    assert lib.sense_read_bandwidth_probe(None, 1024, p(FAKE), None) == INVALID
    assert lib.sense_read_bandwidth_probe(p(FAKE), 0, p(FAKE), None) == INVALID
    assert lib.sense_read_bandwidth_probe(p(FAKE + 8), 1024, p(FAKE), None) == MISALIGNED
    assert lib.sense_read_bandwidth_probe(p(FAKE), 1000, p(FAKE), None) == MISALIGNED


def test_verify_empty_batch_is_a_no_op(lib):
    assert verify_call(lib, n_cand=0, logits=None, drafts=None, acc=None, best=None, ws=None) == 0


def test_verify_workspace_size(lib):
    size = ctypes.c_size_t()
    assert lib.sense_soft_gate_verify_workspace_size(64, 8, 152064, ctypes.byref(size)) == 0
    assert size.value >= 64 * 8 * 16                 # one 16-byte partial per row at least
    assert lib.sense_soft_gate_verify_workspace_size(8, 65, 100, ctypes.byref(size)) == INVALID
    assert lib.sense_soft_gate_verify_workspace_size(8, 8, 100, None) == INVALID


def test_binding_refuses_host_tensors():
    import torch
    keys = torch.zeros(16, 8, dtype=torch.bfloat16)
    spans = torch.zeros(16, 4, dtype=torch.int32)
    with pytest.raises(ValueError):
        sense.sense_build_index(keys, spans)
    with pytest.raises(ValueError):
        sense.sense_soft_gate_verify(torch.zeros(2, 3, 10), torch.zeros(2, 3, dtype=torch.int32))


def dyn_desc(**kw):
    base = dict(key_dtype=sense.SENSE_BF16, d=256, capacity=4096, max_span=8, metric=1)
    base.update(kw)
    return sense.DynamicIndexDesc(**base)


@pytest.mark.parametrize("kw", [
    dict(key_dtype=sense.SENSE_F32),
    dict(d=0), dict(d=100), dict(d=8200),
    dict(capacity=0), dict(capacity=1 << 31),
    dict(max_span=0), dict(max_span=65),
    dict(metric=3),
])
def test_build_dynamic_index_rejects(lib, kw):
    out = ctypes.c_void_p(123)
    d = dyn_desc(**kw)
    assert lib.sense_build_dynamic_index(ctypes.byref(d), ctypes.byref(out)) == INVALID
    assert out.value is None
    assert lib.sense_last_error_message()


def test_dynamic_index_null_args(lib):
    out = ctypes.c_void_p()
    assert lib.sense_build_dynamic_index(None, ctypes.byref(out)) == INVALID
    d = dyn_desc()
    assert lib.sense_build_dynamic_index(ctypes.byref(d), None) == INVALID
    assert lib.sense_index_append(None, p(FAKE), 0, p(FAKE), 4, None) == INVALID


def select_call(lib, **kw):
    a = dict(ss=p(FAKE), ds=p(FAKE), ls=None, ns=64, sd=p(FAKE), dd=p(FAKE), ld=None, nd=16,
             anchors=p(FAKE), nq=1, m=8, top_n=32,
             params=sense.SelectParams(alpha=100.0, beta=1.0, delta=0.1, anchor_override=1),
             od=p(FAKE), ol=p(FAKE), osrc=None, osc=None)
    a.update(kw)
    prm = a["params"]
    return lib.sense_select_candidates(
        a["ss"], a["ds"], a["ls"], a["ns"], a["sd"], a["dd"], a["ld"], a["nd"], a["anchors"],
        a["nq"], a["m"], a["top_n"], None if prm is None else ctypes.byref(prm), a["od"],
        a["ol"], a["osrc"], a["osc"], None)


NAN = float("nan")


@pytest.mark.parametrize("kw,status", [
    (dict(params=None), INVALID),
    (dict(ns=-1), INVALID),
    (dict(nd=-1), INVALID),
    (dict(ns=0, nd=0, top_n=1), INVALID),
    (dict(ns=2000, nd=49), UNSUPPORTED),
    (dict(top_n=0), INVALID),
    (dict(top_n=81), INVALID),
    (dict(m=0), INVALID),
    (dict(m=65), INVALID),
    (dict(nq=0), INVALID),
    (dict(ss=None), INVALID),
    (dict(ds=None), INVALID),
    (dict(sd=None), INVALID),
    (dict(dd=None), INVALID),
    (dict(anchors=None), INVALID),
    (dict(od=None), INVALID),
    (dict(ol=None), INVALID),
    (dict(params=sense.SelectParams(alpha=NAN, beta=1.0, delta=0.0, anchor_override=1)), INVALID),
    (dict(params=sense.SelectParams(alpha=1.0, beta=NAN, delta=0.0, anchor_override=1)), INVALID),
    (dict(params=sense.SelectParams(alpha=1.0, beta=1.0, delta=NAN, anchor_override=1)), INVALID),
])
def test_select_rejects(lib, kw, status):
    assert select_call(lib, **kw) == status
    assert lib.sense_last_error_message()


def test_timer_ids(lib):
    assert lib.sense_set_timer_events(sense.SENSE_TIMER_SELECT, None, None) == 0
    assert lib.sense_set_timer_events(sense.SENSE_TIMER_TRIE, None, None) == 0
    assert lib.sense_set_timer_events(sense.SENSE_TIMER_PROJECT, None, None) == 0
    assert lib.sense_set_timer_events(sense.SENSE_TIMER_IVF, None, None) == 0
    assert lib.sense_set_timer_events(sense.SENSE_TIMER_FILTER, None, None) == 0
    assert lib.sense_set_timer_events(8, None, None) == INVALID


def trie_desc(**kw):
    base = dict(order=p(FAKE), gamma=p(FAKE), tree_tokens=p(FAKE), tree_parent=p(FAKE),
                tree_depth=p(FAKE), tree_cand=p(FAKE), tree_len=p(FAKE), sorted_drafts=None,
                sorted_len=None, mask=None, mask_ld=0, full_mask=None, full_mask_dtype=0,
                prefix_len=0, cache_len=0)
    base.update(kw)
    return sense.TrieDesc(**base)


@pytest.mark.parametrize("args,kw,status", [
    (dict(n_cand=0), {}, INVALID),
    (dict(max_len=0), {}, INVALID),
    (dict(max_len=65), {}, INVALID),
    (dict(n_groups=3), {}, INVALID),                 # 64 % 3 != 0
    (dict(n_groups=0), {}, INVALID),
    (dict(n_cand=2048, n_groups=1, max_len=1), {}, UNSUPPORTED),   # > 1024 drafts
    (dict(n_cand=128, max_len=64), {}, UNSUPPORTED),               # > 4096 tokens
    (dict(drafts=None), {}, INVALID),
    ({}, dict(order=None), INVALID),
    ({}, dict(gamma=None), INVALID),
    ({}, dict(tree_tokens=None), INVALID),
    ({}, dict(tree_parent=None), INVALID),
    ({}, dict(tree_depth=None), INVALID),
    ({}, dict(tree_cand=None), INVALID),
    ({}, dict(tree_len=None), INVALID),
    ({}, dict(mask=p(FAKE), mask_ld=100), INVALID),               # < 512 nodes
    ({}, dict(full_mask=p(FAKE), full_mask_dtype=9, cache_len=10), INVALID),
    ({}, dict(full_mask=p(FAKE), full_mask_dtype=0, cache_len=0), INVALID),
    ({}, dict(full_mask=p(FAKE), full_mask_dtype=0, prefix_len=-1, cache_len=10), INVALID),
    ({}, dict(full_mask=p(FAKE + 2), full_mask_dtype=0, cache_len=10), MISALIGNED),
])
def test_trie_rejects(lib, args, kw, status):
    a = dict(drafts=p(FAKE), dl=None, n_cand=64, max_len=8, n_groups=1)
    a.update(args)
    d = trie_desc(**kw)
    assert lib.sense_build_loose_trie(a["drafts"], a["dl"], a["n_cand"], a["max_len"],
                                      a["n_groups"], ctypes.byref(d), None) == status
    assert lib.sense_last_error_message()
    assert lib.sense_build_loose_trie(p(FAKE), None, 64, 8, 1, None, None) == INVALID


def tree_verify_call(lib, **kw):
    a = dict(logits=p(FAKE), dtype=0, row_stride=1000, tok=p(FAKE), par=p(FAKE), tl=p(FAKE),
             gam=p(FAKE), n_cand=8, max_len=8, vocab=1000, n_groups=1,
             params=sense.GateParams(gamma=0.05, topk=3, window=6, tau=0, entropy_normalized=1),
             acc=p(FAKE), best=p(FAKE), ws=p(FAKE), ws_bytes=1 << 30)
    a.update(kw)
    prm = a["params"]
    return lib.sense_soft_gate_verify_tree(
        a["logits"], a["dtype"], a["row_stride"], a["tok"], a["par"], a["tl"], a["gam"],
        a["n_cand"], a["max_len"], a["vocab"], a["n_groups"],
        None if prm is None else ctypes.byref(prm), a["acc"], a["best"], None, None, None,
        a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(params=None), INVALID),
    (dict(n_cand=-1), INVALID),
    (dict(max_len=0), INVALID),
    (dict(vocab=0), INVALID),
    (dict(row_stride=999), INVALID),
    (dict(dtype=5), INVALID),
    (dict(n_groups=3), INVALID),
    (dict(n_cand=2048, max_len=1), UNSUPPORTED),
    (dict(logits=None), INVALID),
    (dict(tok=None), INVALID),
    (dict(par=None), INVALID),
    (dict(tl=None), INVALID),
    (dict(gam=None), INVALID),
    (dict(acc=None), INVALID),
    (dict(best=None), INVALID),
    (dict(ws=None), WORKSPACE),
    (dict(ws_bytes=16), WORKSPACE),
    (dict(ws=p(FAKE + 64)), MISALIGNED),
    (dict(logits=p(FAKE + 2)), MISALIGNED),
])
def test_tree_verify_rejects(lib, kw, status):
    assert tree_verify_call(lib, **kw) == status
    assert lib.sense_last_error_message()


def test_tree_verify_empty_and_workspace(lib):
    assert tree_verify_call(lib, n_cand=0, logits=None, tok=None, ws=None) == 0
    size = ctypes.c_size_t()
    assert lib.sense_soft_gate_verify_tree_workspace_size(64, 8, 152064, 1, ctypes.byref(size)) == 0
    assert size.value >= 64 * 8 * 16
    assert lib.sense_soft_gate_verify_tree_workspace_size(64, 8, 100, 3,
                                                         ctypes.byref(size)) == INVALID


def proj(**kw):
    base = dict(mean=None, basis=p(FAKE), d_in=4096, d_out=64, normalize=1)
    base.update(kw)
    return sense.ProjDesc(**base)


@pytest.mark.parametrize("kw,args,status", [
    (dict(basis=None), {}, INVALID),
    (dict(d_in=0), {}, INVALID),
    (dict(d_in=100), {}, INVALID),
    (dict(d_in=8200), {}, INVALID),
    (dict(d_out=0), {}, INVALID),
    (dict(d_out=257), {}, INVALID),
    (dict(basis=p(FAKE + 2)), {}, MISALIGNED),
    ({}, dict(xdt=7), INVALID),
    ({}, dict(odt=7), INVALID),
    ({}, dict(n=-1), INVALID),
    ({}, dict(xs=4000), INVALID),
    ({}, dict(os=10), INVALID),
    ({}, dict(x=None), INVALID),
    ({}, dict(out=None), INVALID),
    ({}, dict(x=p(FAKE + 1), xdt=2), MISALIGNED),
    ({}, dict(ws=None), WORKSPACE),                  # 16-bit, aligned, 1000 rows: MFMA route
    ({}, dict(wsb=64), WORKSPACE),
    ({}, dict(ws=p(FAKE + 64)), MISALIGNED),
])
def test_project_rejects(lib, kw, args, status):
    a = dict(x=p(FAKE), xdt=sense.SENSE_BF16, n=1000, xs=4096, out=p(FAKE), odt=sense.SENSE_BF16,
             os=64, ws=p(FAKE), wsb=1 << 30)
    a.update(args)
    d = proj(**kw)
    assert lib.sense_project(ctypes.byref(d), a["x"], a["xdt"], a["n"], a["xs"], a["out"],
                             a["odt"], a["os"], a["ws"], a["wsb"], None) == status
    assert lib.sense_last_error_message()


def test_project_workspace_sizes(lib):
    size = ctypes.c_size_t()
    d = proj()
    assert lib.sense_project_workspace_size(ctypes.byref(d), sense.SENSE_BF16, 1 << 20,
                                            ctypes.byref(size)) == 0
    # matrix-core route, up to 64 outputs: centring and normalisation in the
    # scan's epilogue, no d_out x n intermediate
    assert 0 < size.value < 64 * (1 << 20) * 4
    wide = proj(d_out=100)
    assert lib.sense_project_workspace_size(ctypes.byref(wide), sense.SENSE_BF16, 1 << 20,
                                            ctypes.byref(size)) == 0
    assert size.value >= 100 * (1 << 20) * 4               # S = d_out x n fp32
    assert lib.sense_project_workspace_size(ctypes.byref(d), sense.SENSE_F32, 1 << 20,
                                            ctypes.byref(size)) == 0
    assert size.value >= 64 * (1 << 20) * 4                # fp32 rows: raw results
    assert lib.sense_project_workspace_size(ctypes.byref(d), sense.SENSE_BF16, 0,
                                            ctypes.byref(size)) == 0
    assert size.value == 0
    assert lib.sense_project(ctypes.byref(d), None, 2, 0, 4096, None, 2, 64, None, 0, None) == 0


# ---------------------------------------------------------------- inverted file

@pytest.mark.parametrize("args,status", [
    (dict(kdt=sense.SENSE_F32), INVALID),
    (dict(n=0), INVALID),
    (dict(d=100), INVALID),          # not a multiple of 8
    (dict(d=136), INVALID),          # above the largest key dimension
    (dict(ks=32), INVALID),          # stride below d
    (dict(keys=p(FAKE + 2)), MISALIGNED),
    (dict(ks=68), MISALIGNED),       # stride % 8 != 0
    (dict(keys=None), INVALID),
    (dict(cen=None), INVALID),
    (dict(out=None), INVALID),
    (dict(nlist=0), INVALID),
    (dict(nlist=65537), INVALID),
    (dict(metric=7), INVALID),
    (dict(cen=p(FAKE + 2)), MISALIGNED),
])
def test_ivf_assign_rejects(lib, args, status):
    a = dict(keys=p(FAKE), kdt=sense.SENSE_BF16, n=1000, d=64, ks=64, cen=p(FAKE), nlist=16,
             metric=1, out=p(FAKE))
    a.update(args)
    assert lib.sense_ivf_assign(a["keys"], a["kdt"], a["n"], a["d"], a["ks"], a["cen"], a["nlist"],
                                a["metric"], a["out"], None) == status
    assert lib.sense_last_error_message()


@pytest.mark.parametrize("args,status", [
    (dict(m=0), INVALID),
    (dict(m=3), INVALID),            # does not divide d = 64
    (dict(m=2), INVALID),            # 32-dim sub-vectors: above 16
    (dict(ksub=0), INVALID),
    (dict(ksub=257), INVALID),
    (dict(d=128, ksub=256), INVALID),   # ksub * d > 16384
    (dict(lists=None), INVALID),
    (dict(books=None), INVALID),
    (dict(out=None), INVALID),
    (dict(nlist=0), INVALID),
    (dict(books=p(FAKE + 2)), MISALIGNED),
    (dict(lists=p(FAKE + 2)), MISALIGNED),
])
def test_pq_encode_rejects(lib, args, status):
    a = dict(keys=p(FAKE), kdt=sense.SENSE_BF16, n=1000, d=64, ks=64, cen=p(FAKE), nlist=16,
             lists=p(FAKE), books=p(FAKE), m=16, ksub=256, out=p(FAKE))
    a.update(args)
    assert lib.sense_pq_encode(a["keys"], a["kdt"], a["n"], a["d"], a["ks"], a["cen"], a["nlist"],
                               a["lists"], a["books"], a["m"], a["ksub"], a["out"], None) == status
    assert lib.sense_last_error_message()


def ivf_desc(**kw):
    base = dict(keys=FAKE, key_dtype=sense.SENSE_BF16, n=1000, d=64, key_stride=64, spans=FAKE,
                max_span=8, span_len=None, metric=1, centroids=FAKE, nlist=16, list_ids=FAKE,
                pq_codebooks=None, pq_m=0, pq_ksub=0, pq_codes=None)
    base.update(kw)
    return sense.IvfDesc(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(d=100), INVALID),
    (dict(n=0), INVALID),
    (dict(keys=None), INVALID),                      # IVF-Flat needs its keys
    (dict(spans=None), INVALID),
    (dict(centroids=None), INVALID),
    (dict(list_ids=None), INVALID),
    (dict(nlist=0), INVALID),
    (dict(nlist=70000), INVALID),
    (dict(max_span=0), INVALID),
    (dict(max_span=65), INVALID),
    (dict(metric=5), INVALID),
    (dict(keys=FAKE + 2), MISALIGNED),
    (dict(pq_codebooks=FAKE, pq_m=16, pq_ksub=256, pq_codes=None, keys=None), INVALID),
    (dict(pq_codebooks=FAKE, pq_m=3, pq_ksub=256, pq_codes=FAKE, keys=None), INVALID),
    (dict(pq_codebooks=FAKE, pq_m=16, pq_ksub=300, pq_codes=FAKE, keys=None), INVALID),
])
def test_build_ivf_index_rejects(lib, kw, status):
    d = ivf_desc(**kw)
    out = ctypes.c_void_p(1234)
    assert lib.sense_build_ivf_index(ctypes.byref(d), None, ctypes.byref(out)) == status
    assert out.value is None                          # cleared before validation fails
    assert lib.sense_last_error_message()


def test_ivf_search_rejects_null_index(lib):
    size = ctypes.c_size_t()
    assert lib.sense_ivf_search_workspace_size(None, 1, 64, 32, ctypes.byref(size)) == INVALID
    assert lib.sense_ivf_search(None, p(FAKE), sense.SENSE_F32, 1, 64, 32, p(FAKE), p(FAKE),
                                None, None, None, p(FAKE), 1 << 20, None) == INVALID
    assert lib.sense_build_ivf_index(None, None, None) == INVALID
