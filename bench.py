#!/usr/bin/env python3
"""Throughput of the SENSE retrieval + soft-gated evaluation hot path on one
MI355X.

One step = one sense_retrieve over the whole datastore (similarity scan,
top-k, gather of the continuations) followed by one sense_soft_gate_verify
of the retrieved drafts of the verified queries against their aligned
logits.  Inputs are synthetic (see paper_2606_00021_amd/synth.py) and
resident in HBM before the timed region starts.  The "sen" object times the
method's full drafting step apart from it: static and dynamic-cache
retrieval, composite Top-N selection, the loose trie and verification
through it.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0   # MI355X HBM3E, published
MFMA_PEAK_TFLOPS = 2500.0   # MI355X dense fp16/bf16 matrix-core peak (published)
METRIC = "retrieval+verify queries/sec and achieved HBM GB/s (% of peak) at N=1M, d=4096"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None, help="workload name (default: the headline)")
    ap.add_argument("--seed", type=int, default=1003)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time spent timing the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--config-cpu-seconds", type=float, default=3.0,
                    help="approximate CPU time for the oracle timing of each other configuration")
    ap.add_argument("--graph", action="store_true",
                    help="also time replays of the step captured as one HIP graph (on this "
                         "ROCm the replays measured a few us slower than eager launches)")
    ap.add_argument("--no-sen", action="store_true",
                    help="skip the candidate-selection leg (dynamic cache + composite Top-N)")
    ap.add_argument("--sen-context", type=int, default=4096,
                    help="rows of generation context in the dynamic cache of the SEN leg")
    ap.add_argument("--no-configs", action="store_true",
                    help="time the headline workload only (by default every other "
                         "configuration of the metric follows it)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the timed region, run one plain device copy of this many MiB "
                         "(a reference kernel of known traffic for HBM counter runs)")
    return ap.parse_args()


def scan_source_digest(fname: str = "scan.hip") -> str:
    """Digest of a scan kernel's source file with comments and blank space
    removed (comment edits do not invalidate measured counters)."""
    import hashlib
    import re

    src = open(os.path.join(ROOT, "paper_2606_00021_amd", "csrc", fname)).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    src = "".join(src.split())
    return hashlib.sha256(src.encode()).hexdigest()[:16]


SCAN_SOURCES = {"scan_gemv_kernel": "scan.hip", "scan_small_kernel": "scan_small.hip",
                "scan_mfma_kernel": "scan_mfma.hip"}


def traffic_from_profiles(workload: str, kernel: str = "scan_gemv_kernel"):
    """Measured HBM bytes per scan launch, read from the committed rocprofv3
    counter summary of this kernel and workload, or None when there is none or
    the kernel's source changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith(("|", "-", "#", "`")):
            key, _, val = line.partition(":")
            fields[key.strip()] = val.strip()
    if (fields.get("scan_source_sha256_16") != scan_source_digest(SCAN_SOURCES[kernel])
            or "bytes_per_launch" not in fields):
        return None
    return int(fields["bytes_per_launch"])


def cpu_baseline(w, ds, q, logits, drafts, budget_s: float, max_sample_bytes=None):
    """The oracle as it stands, timed on this host on a bounded sample of the
    same workload, scaled to one query (its scan + sort + gather + verify)."""
    import numpy as np
    import torch

    import oracle

    cores = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or os.cpu_count()
    kb_dt = w.key_dtype
    qh = q.cpu().numpy()
    # Calibrate the scan on a small block, then size the sample to the budget.
    cal = 2048
    keys_cal = ds.keys[:cal].cpu().view(torch.int16).numpy().view(np.uint16)
    t0 = time.perf_counter()
    oracle.scores(keys_cal, kb_dt, qh[:1], "f32", metric=w.metric)
    per_row = (time.perf_counter() - t0) / cal
    rows = int(min(w.n, max(cal, 0.6 * budget_s / max(per_row, 1e-9))))
    if max_sample_bytes is not None:          # keys copied to the host for the sample
        rows = max(cal, min(rows, int(max_sample_bytes // (ds.keys.shape[1] * 2))))
    keys_s = ds.keys[:rows].cpu().view(torch.int16).numpy().view(np.uint16)
    t0 = time.perf_counter()
    oracle.scores(keys_s, kb_dt, qh[:1], "f32", metric=w.metric)
    t_scan_row = (time.perf_counter() - t0) / rows
    # Full sort of N scores (the oracle's top-k) and the gather.
    rng = np.random.default_rng(0)
    fake = rng.standard_normal(w.n)
    t0 = time.perf_counter()
    ids, _ = oracle.topk(fake, w.k)
    oracle.gather(ds.spans[:1024].cpu().numpy(), None, ids % 1024)
    t_sort = time.perf_counter() - t0
    # Verify: a sample of candidates, scaled per position.
    dt_name = {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[logits.dtype]
    c_s = max(1, min(drafts.shape[0], 8))
    lg = logits[:c_s].cpu()
    lg = lg.view(torch.int16).numpy().view(np.uint16) if dt_name != "f32" else lg.numpy()
    t0 = time.perf_counter()
    oracle.soft_gate_verify(lg, dt_name, drafts[:c_s].cpu().numpy())
    t_verify_pos = (time.perf_counter() - t0) / (c_s * drafts.shape[1])
    pos_per_query = w.n_cand * w.span / w.n_queries
    t_query = t_scan_row * w.n + t_sort + t_verify_pos * pos_per_query
    # The same oracle on one core (its OpenMP loops on one thread), on a
    # sample as many times smaller as there are cores; the sort is one thread
    # in both.
    prev = oracle.set_threads(1)
    try:
        rows1 = max(cal, rows // max(1, cores))
        t0 = time.perf_counter()
        oracle.scores(keys_s[:rows1], kb_dt, qh[:1], "f32", metric=w.metric)
        t_scan_row1 = (time.perf_counter() - t0) / rows1
        t0 = time.perf_counter()
        oracle.soft_gate_verify(lg[:1], dt_name, drafts[:1].cpu().numpy())
        t_verify_pos1 = (time.perf_counter() - t0) / drafts.shape[1]
    finally:
        oracle.set_threads(prev)
    t_query1 = t_scan_row1 * w.n + t_sort + t_verify_pos1 * pos_per_query
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")),
                             None)
    except OSError:
        pass
    return {
        "value": 1.0 / t_query,
        "unit": "queries/s",
        "cores": cores,
        "cpu_model": cpu_model,
        "kind": "oracle",
        "sample": (f"fp64 oracle on host: scan of {rows} of {w.n} rows x d={ds.keys.shape[1]} "
                   f"({t_scan_row * 1e6:.3f} us/row), full sort of {w.n} scores "
                   f"({t_sort:.3f} s), verify of {c_s}x{drafts.shape[1]} positions x "
                   f"V={w.vocab} ({t_verify_pos * 1e3:.2f} ms/position); scaled to one "
                   f"query = {w.n} rows + sort + {pos_per_query:.0f} positions"),
        "value_1core": 1.0 / t_query1,
        "sample_1core": (f"the same oracle on one thread: scan of {rows1} rows "
                         f"({t_scan_row1 * 1e6:.3f} us/row), verify of 1x{drafts.shape[1]} "
                         f"positions ({t_verify_pos1 * 1e3:.2f} ms/position), the same sort; "
                         f"scaled to one query alike"),
    }


def sen_leg(args, w, ds, q, src_rows, K, dev):
    """The paper's full drafting + verification step, timed apart from the
    headline step: static retrieval (k hits) over the same keys with
    continuations that overlap between neighbours, dynamic-cache retrieval
    over a generation context, composite Top-N (alpha 100, beta 1, delta 0.05,
    anchor override), LexSort + loose trie of the N drafts, and verification
    through Gamma.  Also times each stage alone, the dense verification of
    the same drafts (one logits row per draft position) and one cache append
    of 4 accepted positions."""
    import torch

    from paper_2606_00021_amd import sense, synth

    k, m, nq = w.k, w.span, w.n_queries
    k_dyn, top_n, ctx_len = 16, w.k, args.sen_context
    spans = synth.make_shared_spans(w, ds, args.seed)
    index = sense.sense_build_index(ds.keys, spans, None, metric=w.metric)
    anchors = spans[src_rows, 0].to(torch.int32).contiguous()
    ctx = synth.make_context(w, ds, args.seed, ctx_len, int(src_rows[0]), int(anchors[0]))
    kdt = synth.DTYPES[w.key_dtype]
    cache = sense.sense_build_dynamic_index(w.d, ctx_len, m, key_dtype=kdt, metric=w.metric)
    sense.sense_index_append(cache, ctx.keys, ctx.tokens)

    def retr_bufs(kk):
        return (torch.empty((nq, kk), dtype=torch.int64, device=dev),
                torch.empty((nq, kk), dtype=torch.float32, device=dev),
                torch.empty((nq, kk, m), dtype=torch.int32, device=dev),
                torch.empty((nq, kk), dtype=torch.int32, device=dev))
    ws_s = torch.empty(max(1, sense.sense_retrieve_workspace_size(index, nq, k)),
                       dtype=torch.uint8, device=dev)
    ws_d = torch.empty(max(1, sense.sense_retrieve_workspace_size(cache, nq, k_dyn)),
                       dtype=torch.uint8, device=dev)
    outs_s, outs_d = retr_bufs(k), retr_bufs(k_dyn)
    sel = (torch.empty((nq, top_n, m), dtype=torch.int32, device=dev),
           torch.empty((nq, top_n), dtype=torch.int32, device=dev),
           torch.empty((nq, top_n), dtype=torch.int32, device=dev),
           torch.empty((nq, top_n), dtype=torch.float32, device=dev))
    vq = w.verify_queries
    c = vq * top_n
    drafts = sel[0][:vq].view(c, m)
    dlen = sel[1][:vq].view(c)

    # The dynamic search is independent of the static one: it runs on a
    # second stream (default priority) while the static scan streams HBM.
    side = torch.cuda.Stream()
    fork, join = torch.cuda.Event(), torch.cuda.Event()

    def draft_stage():
        main_stream = torch.cuda.current_stream()
        fork.record(main_stream)
        side.wait_event(fork)
        sense.sense_retrieve(cache, q, k_dyn, workspace=ws_d, out=outs_d, stream=side)
        join.record(side)
        sense.sense_retrieve(index, q, k, workspace=ws_s, out=outs_s)
        main_stream.wait_event(join)
        sense.sense_select_candidates((outs_s[1], outs_s[2], outs_s[3]),
                                      (outs_d[1], outs_d[2], outs_d[3]), anchors, top_n,
                                      100.0, 1.0, 0.05, True, out=sel)

    draft_stage()
    tr = sense.sense_build_loose_trie(drafts, dlen, n_groups=vq)
    torch.cuda.synchronize()
    nodes = top_n * m
    tl = tr["tree_len"].cpu().numpy()
    logits = synth.make_tree_logits(w.vocab, w.logits_dtype, vq, nodes,
                                    tr["tree_tokens"].cpu().numpy(),
                                    tr["tree_parent"].cpu().numpy(), tl, args.seed + 1, dev)
    ws_v = torch.empty(max(1, sense.sense_soft_gate_verify_tree_workspace_size(c, m, w.vocab, vq)),
                       dtype=torch.uint8, device=dev)
    out_v = {"accept_len": torch.empty(c, dtype=torch.int32, device=dev),
             "best": torch.empty(vq, dtype=torch.int32, device=dev)}
    # Dense comparison: the same aligned rows copied out, one per position.
    gam = tr["gamma"].long().view(vq, top_n, m)
    rows = torch.zeros_like(gam)
    rows[..., 1:] = torch.where(gam[..., :-1] >= 0, gam[..., :-1] + 1, torch.zeros_like(gam[..., :-1]))
    dense = torch.stack([logits[g][rows[g]] for g in range(vq)]).view(c, m, w.vocab).contiguous()
    sdr, sln = tr["sorted_drafts"], tr["sorted_len"]
    ws_dv = torch.empty(max(1, sense.sense_soft_gate_verify_workspace_size(c, m, w.vocab)),
                        dtype=torch.uint8, device=dev)
    out_dv = {"accept_len": torch.empty(c, dtype=torch.int32, device=dev),
              "best": torch.empty(vq, dtype=torch.int32, device=dev)}

    def step():
        draft_stage()
        sense.sense_build_loose_trie(drafts, dlen, n_groups=vq, out=tr)
        sense.sense_soft_gate_verify_tree(logits, tr, n_groups=vq, workspace=ws_v, out=out_v)

    def timed(fn, reps):
        for _ in range(3):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    ms_step = timed(step, K)

    # Per-stage kernel durations: hipEvents recorded by the library around
    # each stage's kernels (a second pass; the host's launch rate does not
    # enter these, unlike back-to-back calls of one small stage).
    def events():
        pair = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        for e in pair:
            e.record()                       # creates the hipEvent
        return pair
    stages = ("dyn_scan", "dyn_topk", "select", "trie", "verify_tree", "verify_dense", "append")
    ev = {t: [events() for _ in range(K)] for t in stages}
    grow = sense.sense_build_dynamic_index(w.d, 4 * (K + 3), m, key_dtype=kdt, metric=w.metric)
    new_keys, new_tok = ctx.keys[:4].contiguous(), ctx.tokens[:4].contiguous()
    torch.cuda.synchronize()
    T = sense
    for i in range(K):
        sense.sense_retrieve(index, q, k, workspace=ws_s, out=outs_s)
        T.sense_set_timer_events(T.SENSE_TIMER_SCAN, *ev["dyn_scan"][i])
        T.sense_set_timer_events(T.SENSE_TIMER_TOPK, *ev["dyn_topk"][i])
        sense.sense_retrieve(cache, q, k_dyn, workspace=ws_d, out=outs_d)
        T.sense_set_timer_events(T.SENSE_TIMER_SCAN, None, None)
        T.sense_set_timer_events(T.SENSE_TIMER_TOPK, None, None)
        T.sense_set_timer_events(T.SENSE_TIMER_SELECT, *ev["select"][i])
        sense.sense_select_candidates((outs_s[1], outs_s[2], outs_s[3]),
                                      (outs_d[1], outs_d[2], outs_d[3]), anchors, top_n,
                                      100.0, 1.0, 0.05, True, out=sel)
        T.sense_set_timer_events(T.SENSE_TIMER_TRIE, *ev["trie"][i])
        sense.sense_build_loose_trie(drafts, dlen, n_groups=vq, out=tr)
        T.sense_set_timer_events(T.SENSE_TIMER_VERIFY, *ev["verify_tree"][i])
        sense.sense_soft_gate_verify_tree(logits, tr, n_groups=vq, workspace=ws_v, out=out_v)
        T.sense_set_timer_events(T.SENSE_TIMER_VERIFY, *ev["verify_dense"][i])
        sense.sense_soft_gate_verify(dense, sdr, sln, n_groups=vq, workspace=ws_dv, out=out_dv)
        T.sense_set_timer_events(T.SENSE_TIMER_VERIFY, None, None)
        a, b = ev["append"][i]
        a.record()
        sense.sense_index_append(grow, new_keys, new_tok)
        b.record()
    torch.cuda.synchronize()
    for t in (T.SENSE_TIMER_SELECT, T.SENSE_TIMER_TRIE):
        T.sense_set_timer_events(t, None, None)
    dur = {t: sum(a.elapsed_time(b) for a, b in ev[t]) / K for t in stages}
    dyn_ms = dur["dyn_scan"] + dur["dyn_topk"]
    sel_ms, trie_ms = dur["select"], dur["trie"]
    vt_ms, vd_ms, append_ms = dur["verify_tree"], dur["verify_dense"], dur["append"]
    grow.close()
    L = int(tl.sum())
    positions = int(sln.clamp(0, m).sum().item())
    ebytes = 4 if w.logits_dtype == "f32" else 2
    cache.close()
    index.close()
    log(f"[bench] SEN step {ms_step:.4f} ms: dynamic retrieval {dyn_ms * 1e3:.1f} us over "
        f"{ctx_len} rows, selection {sel_ms * 1e3:.1f} us, trie {trie_ms * 1e3:.1f} us "
        f"({L} nodes for {positions} draft tokens), verify through the tree "
        f"{vt_ms * 1e3:.1f} us vs dense {vd_ms * 1e3:.1f} us, append {append_ms * 1e3:.1f} us")
    return {"queries_per_s": nq / (ms_step * 1e-3), "ms_per_step": ms_step,
            "context_rows": ctx_len, "k_static": k, "k_dynamic": k_dyn, "top_n": top_n,
            "alpha": 100.0, "beta": 1.0, "delta": 0.05,
            "dynamic_retrieve_us": dyn_ms * 1e3, "select_us": sel_ms * 1e3,
            "trie_us": trie_ms * 1e3, "tree_nodes": L, "draft_tokens": positions,
            "tree_fraction": L / max(positions, 1),
            "verify_tree_us": vt_ms * 1e3, "verify_dense_us": vd_ms * 1e3,
            "verify_tree_gbps": L * w.vocab * ebytes / (vt_ms * 1e-3) / 1e9,
            "append4_us": append_ms * 1e3}


# The configurations the metric's workload is quoted beside: besides the
# headline, the tiny store, the LLaMA-3-8B and Qwen2-7B shapes (one query),
# and the 13B-shaped (16 queries) and 70B-shaped (64 queries) batches.
CONFIG_WORKLOADS = ["tiny-16k-d4096", "llama3-8b-262k-d4096", "qwen2-7b-1m-d3584",
                    "13b-batched-4m-d5120", "70b-8m-d8192"]
BATCH_DIRECT_MAX = 131072    # larger stores take the sampled-threshold batched search


def run_workload(name, args, dev, K, warmup, graph=False, copy_probe_mib=0):
    """Builds workload `name`, times K steps after `warmup` untimed ones and
    returns (result dict, context for the SEN leg and the CPU baseline)."""
    import torch

    from paper_2606_00021_amd import sense, synth

    w = synth.WORKLOADS[name]
    log(f"[bench] workload {name}: n={w.n} d={w.d} {w.key_dtype} Q={w.n_queries} k={w.k} "
        f"M={w.span} V={w.vocab} {w.logits_dtype}")
    t0 = time.perf_counter()
    ds = synth.make_datastore(w, args.seed, dev)
    q, src_rows = synth.make_queries(w, ds, args.seed)
    nq, k, m = w.n_queries, w.k, w.span
    proj_info = None
    q_hidden = q
    if w.proj:
        # The paper's key geometry: PCA 4096 -> proj, L2-normalised, stored in
        # the key type.  Projecting the store is the datastore build (timed
        # here, outside the step); the query is projected inside every step.
        mean, basis = synth.make_pca_basis(ds, args.seed, w.proj)
        kdt = synth.DTYPES[w.key_dtype]
        ws_p = torch.empty(max(1, sense.sense_project_workspace_size(basis, kdt, w.n, mean)),
                           dtype=torch.uint8, device=dev)
        keys_p = torch.empty((w.n, w.proj), dtype=kdt, device=dev)
        sense.sense_project(ds.keys, basis, mean, True, out=keys_p, workspace=ws_p)
        torch.cuda.synchronize()
        a_ev, b_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a_ev.record()
        sense.sense_project(ds.keys, basis, mean, True, out=keys_p, workspace=ws_p)
        b_ev.record()
        torch.cuda.synchronize()
        build_ms = a_ev.elapsed_time(b_ev)
        proj_info = {"dim": w.proj, "basis": "top principal directions of a 16384-row sample",
                     "store_projection_ms": build_ms,
                     "store_projection_gbps": w.n * w.d * 2 / (build_ms * 1e-3) / 1e9}
        log(f"[bench] projected the store {w.d} -> {w.proj}: {build_ms:.2f} ms "
            f"({proj_info['store_projection_gbps']:.0f} GB/s of hidden states)")
        del ws_p
        ds.keys = keys_p                      # the searched datastore
        torch.cuda.empty_cache()
        q_proj = torch.empty((nq, w.proj), dtype=torch.float32, device=dev)
        q = q_proj
    d_idx = ds.keys.shape[1]
    index = sense.sense_build_index(ds.keys, ds.spans, ds.span_len, metric=w.metric)
    ivf = None
    ivf_info = None
    if w.ivf_nlist:
        # The paper's ANN retriever over the projected keys.  Training (the
        # k-means fits) is input preparation; assignment, encoding and the
        # list layout are the library's build, timed here.
        cen, books = synth.fit_ivf(ds.keys, args.seed, w.ivf_nlist, pq_m=w.pq_m)
        torch.cuda.synchronize()
        tb = time.perf_counter()
        lists = sense.sense_ivf_assign(ds.keys, cen, w.metric)
        codes = sense.sense_pq_encode(ds.keys, cen, lists, books) if w.pq_m else None
        ivf = sense.sense_build_ivf_index(None if w.pq_m else ds.keys, ds.spans, cen, lists,
                                          ds.span_len, metric=w.metric,
                                          codebooks=books if w.pq_m else None, codes=codes,
                                          key_dtype=ds.keys.dtype)
        torch.cuda.synchronize()
        ivf_info = {"nlist": w.ivf_nlist, "nprobe": w.ivf_nprobe, "pq_m": w.pq_m,
                    "pq_ksub": 256 if w.pq_m else None,
                    "kind": "ivf-pq" if w.pq_m else "ivf-flat",
                    "build_s": time.perf_counter() - tb}
        log(f"[bench] inverted file {ivf_info['kind']} nlist={w.ivf_nlist}: assignment, "
            f"encoding and layout {ivf_info['build_s']:.2f} s")
    if ivf is not None:
        ws_r = torch.empty(max(1, sense.sense_ivf_search_workspace_size(ivf, nq, k, w.ivf_nprobe)),
                           dtype=torch.uint8, device=dev)
    else:
        ws_r = torch.empty(max(1, sense.sense_retrieve_workspace_size(index, nq, k)),
                           dtype=torch.uint8, device=dev)

    def retrieve():
        if ivf is not None:
            sense.sense_ivf_search(ivf, q, k, w.ivf_nprobe, workspace=ws_r, out=outs)
        else:
            sense.sense_retrieve(index, q, k, workspace=ws_r, out=outs)
    outs = (torch.empty((nq, k), dtype=torch.int64, device=dev),
            torch.empty((nq, k), dtype=torch.float32, device=dev),
            torch.empty((nq, k, m), dtype=torch.int32, device=dev),
            torch.empty((nq, k), dtype=torch.int32, device=dev))
    if w.proj:
        sense.sense_project(q_hidden, basis, mean, True, out=q_proj)
    retrieve()
    if ivf is not None:
        # recall@k of the approximate search against the exact scan of the
        # same (projected) keys, over this step's queries
        ex = sense.sense_retrieve(index, q, k)[0]
        torch.cuda.synchronize()
        hits = sum(len(set(outs[0][i].tolist()) & set(ex[i].tolist())) for i in range(nq))
        ivf_info["recall_at_k"] = hits / (nq * k)
        log(f"[bench] recall@{k} against the exact scan: {ivf_info['recall_at_k']:.4f}")
    vq = w.verify_queries
    drafts = outs[2][:vq].view(vq * k, m)
    dlen = outs[3][:vq].view(vq * k)
    logits = synth.make_logits(w, drafts, args.seed)
    c = vq * k
    ws_v = torch.empty(max(1, sense.sense_soft_gate_verify_workspace_size(c, m, w.vocab)),
                       dtype=torch.uint8, device=dev)
    out_v = {"accept_len": torch.empty(c, dtype=torch.int32, device=dev),
             "best": torch.empty(vq, dtype=torch.int32, device=dev)}
    torch.cuda.synchronize()
    log(f"[bench] setup {time.perf_counter() - t0:.1f} s")

    def step():
        if w.proj:
            sense.sense_project(q_hidden, basis, mean, True, out=q_proj)
        retrieve()
        sense.sense_soft_gate_verify(logits, drafts, dlen, n_groups=vq, gamma=0.05, topk=3,
                                     window=6, tau=0, workspace=ws_v, out=out_v)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()

    def time_steps(run):
        # Timed region: exactly K steps between two events, nothing else
        # enqueued.
        t_begin = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        t_begin.record()
        for _ in range(K):
            run()
        t_end.record()
        torch.cuda.synchronize()
        return t_begin.elapsed_time(t_end) / K, (time.perf_counter() - wall0) / K

    ms_eager, wall_eager = time_steps(step)
    ms_step, wall_step = ms_eager, wall_eager
    launch = "eager"
    if graph:
        # The step as one HIP graph: every entry point allocates nothing and
        # records no memset, so the captured kernels replay the same work
        # without the host's per-call launch cost.
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            with torch.cuda.graph(graph, stream=cap):
                step()
        torch.cuda.current_stream().wait_stream(cap)
        graph.replay()
        torch.cuda.synchronize()
        ms_step, wall_step = time_steps(graph.replay)
        launch = "hip_graph"
    wall = wall_step

    # Per-kernel durations: a second pass of K steps with hipEvents recorded
    # by the library around the scan, top-k and verify kernels (the events
    # themselves add a little time, so this pass is not the step time).
    # A batch of long keys over a sampled store: the filtered full pass is
    # the dominant kernel; its own events time it for the roofline.
    filtered = (ivf is None and nq >= 2 and d_idx > 64 and w.n > BATCH_DIRECT_MAX)
    timed_parts = ((("ivf",) if ivf is not None else ("scan", "topk")) + ("verify",)
                   + (("project",) if w.proj else ()) + (("filter",) if filtered else ()))
    ev = {t: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(K)] for t in timed_parts}
    timer_id = {"scan": sense.SENSE_TIMER_SCAN, "topk": sense.SENSE_TIMER_TOPK,
                "filter": sense.SENSE_TIMER_FILTER,
                "verify": sense.SENSE_TIMER_VERIFY, "project": sense.SENSE_TIMER_PROJECT,
                "ivf": sense.SENSE_TIMER_IVF}
    # torch creates the underlying hipEvent_t lazily at the first record():
    # record every event once here so that the handles exist.
    for t in ev:
        for a, b in ev[t]:
            a.record()
            b.record()
    torch.cuda.synchronize()
    for i in range(K):
        for t in ev:
            sense.sense_set_timer_events(timer_id[t], *ev[t][i])
        step()
    torch.cuda.synchronize()
    for t in ev:
        sense.sense_set_timer_events(timer_id[t], None, None)
    dur = {t: sum(a.elapsed_time(b) for a, b in ev[t]) / K for t in ev}
    parts = (f"inverted-file search {dur['ivf']:.4f} ms" if ivf is not None
             else f"scan {dur['scan']:.4f} ms, topk {dur['topk']:.4f} ms")
    if filtered:
        parts += f" (filtered pass {dur['filter']:.4f} ms)"
    log(f"[bench] {K} steps ({launch}): {ms_step:.4f} ms/step (wall {wall * 1e3:.4f} ms/step; "
        f"eager launches {ms_eager:.4f} ms/step); {parts}, verify {dur['verify']:.4f} ms"
        + (f", query projection {dur['project']:.4f} ms" if w.proj else ""))

    # Algorithmic bytes: every key once (+ the fp32 inverse-norm table for
    # cosine), the gathered continuations, and every live logit row once.
    cos_extra = 4 * w.n if w.metric == "cosine" else 0
    scan_bytes = w.n * d_idx * 2 + cos_extra
    gather_bytes = nq * k * m * 4
    live = int(dlen.clamp(0, m).sum().item())
    verify_bytes = live * w.vocab * (4 if w.logits_dtype == "f32" else 2)
    if ivf is not None:
        # Bytes one search must read: the centroids, and per query the probed
        # rows (codes, or keys + norms) of the lists actually probed.
        sizes = torch.bincount(lists.long(), minlength=w.ivf_nlist)
        probe_rows = 0
        for i in range(nq):
            sc_c = q[i].float() @ cen.T
            if w.metric == "cosine":
                sc_c = sc_c / cen.norm(dim=1).clamp_min(1e-30)
            probe_rows += int(sizes[torch.topk(sc_c, w.ivf_nprobe).indices].sum().item())
        row_bytes = w.pq_m if w.pq_m else d_idx * 2 + (4 if w.metric == "cosine" else 0)
        scan_bytes = w.ivf_nlist * d_idx * 4 + probe_rows * (row_bytes + 4)
        ivf_info["probed_rows_per_query"] = probe_rows / nq
        scan_ms = dur["ivf"]
        scan_kernel = "ivf_search"
    else:
        scan_ms = dur["scan"]
        if nq >= 2 and d_idx <= 64:
            # The library's scan events wrap the whole batched short-key
            # retrieval: query split, sample pass, sample top-k, thresholds,
            # filtered pass over every row and the survivors' top-k.
            scan_kernel = "short_key_retrieval"
        elif nq >= 2:
            scan_kernel = "scan_mfma_kernel"
            if filtered:
                # The roofline is the filtered full pass's own: one launch
                # that reads every key (and norm) once.
                scan_ms = dur["filter"]
        elif d_idx <= 64:
            scan_kernel = "scan_small_kernel"
        else:
            scan_kernel = "scan_gemv_kernel"
    step_bytes = scan_bytes + gather_bytes + verify_bytes
    traffic = traffic_from_profiles(name, scan_kernel) if scan_kernel in SCAN_SOURCES else None
    scan_gbps = scan_bytes / (scan_ms * 1e-3) / 1e9
    res = {
        "metric": METRIC,
        "value": nq / (ms_step * 1e-3),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": warmup,
        "ms_per_step": ms_step,
        "launch": launch,
        "ms_per_step_eager": ms_eager,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": name, "n": w.n, "d": w.d, "key_dtype": w.key_dtype,
                   "n_queries": nq, "k": k, "span": m, "vocab": w.vocab,
                   "logits_dtype": w.logits_dtype, "verify_candidates": c,
                   "metric": w.metric, "parallelism": "single-gpu"},
        "hbm_gbps": step_bytes / (ms_step * 1e-3) / 1e9,
        "hbm_frac": step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        **({"ivf_search_ms": dur["ivf"]} if ivf is not None
           else {"scan_ms": dur["scan"], "topk_ms": dur["topk"]}),
        **({"filter_ms": dur["filter"],
            "retrieval_scan_gbps": scan_bytes / (dur["scan"] * 1e-3) / 1e9} if filtered else {}),
        "verify_ms": dur["verify"],
        **({"project_ms": dur["project"]} if w.proj else {}),
        "verify_gbps": verify_bytes / (dur["verify"] * 1e-3) / 1e9 if dur["verify"] > 0 else None,
        "roofline": {"bound": "hbm", "kernel": scan_kernel,
                     **({"timed": "every kernel of the retrieval (scan, selection, gather)"}
                        if scan_kernel in ("short_key_retrieval", "ivf_search") else {}),
                     **({"timed": "the filtered full pass alone (one launch over every row); "
                                  "scan_ms adds the query split and the strided sample's pass "
                                  "and top-k, topk_ms the survivors' selection"}
                        if filtered else {}),
                     "achieved": scan_gbps,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": scan_gbps / HBM_PEAK_GBPS,
                     "traffic": traffic},
    }
    if traffic is not None:
        res["roofline"]["traffic_source"] = (
            f"profiles/{scan_kernel}_{name}.md: rocprofv3 FETCH_SIZE + WRITE_SIZE per launch, "
            f"each scaled by what the counter reads for a 1 GiB device copy; taken on the "
            f"current kernel source (its digest matches), not in this run")
    if scan_kernel == "scan_mfma_kernel":
        # Matrix-core utilisation of the batched scan (bound by HBM, so a share
        # of the dense peak, reported beside GB/s): the instructions issue
        # whole 16-query tiles and 32-dimension steps, twice with fp32 queries
        # (hi + lo halves in the key type) except in a cosine filtered pass,
        # which takes the hi half alone and rescores a band in fp32.
        qpad = 16 * ((nq + 15) // 16)
        dpad = 32 * ((d_idx + 31) // 32)
        halves = 2 if (q.dtype == torch.float32
                       and not (filtered and w.metric == "cosine")) else 1
        issued = 2.0 * w.n * dpad * qpad * halves
        res["mfma"] = {"dtype": w.key_dtype, "issued_flops": issued,
                       "useful_flops": 2.0 * w.n * d_idx * nq,
                       "achieved_tflops": issued / (scan_ms * 1e-3) / 1e12,
                       "peak_tflops": MFMA_PEAK_TFLOPS,
                       "frac": issued / (scan_ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS}
    if ivf_info is not None:
        res["config"]["ivf"] = ivf_info["kind"]
        res["ivf"] = ivf_info
    if proj_info is not None:
        res["config"]["proj"] = w.proj
        res["projection"] = proj_info
    # Practical HBM read ceiling: a plain streaming read of the key store.
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    sense.sense_read_bandwidth_probe(ds.keys, sink)
    probe_ms = []
    for _ in range(5):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        sense.sense_read_bandwidth_probe(ds.keys, sink)
        b.record()
        torch.cuda.synchronize()
        probe_ms.append(a.elapsed_time(b))
    ceiling = ds.keys.numel() * 2 / (min(probe_ms) * 1e-3) / 1e9
    res["hbm_read_ceiling_gbps"] = ceiling
    res["scan_frac_of_read_ceiling"] = scan_gbps / ceiling
    log(f"[bench] plain streaming read of the keys: {ceiling:.0f} GB/s; scan at "
        f"{scan_gbps / ceiling * 100:.1f} % of it")
    if copy_probe_mib > 0:
        n_el = copy_probe_mib * (1 << 20) // 4
        src = torch.ones(n_el, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copy probe: {copy_probe_mib} MiB read + {copy_probe_mib} MiB "
            f"written by one copy kernel")
        del src, dst
    ctx = {"w": w, "ds": ds, "q": q, "src_rows": src_rows, "logits": logits, "drafts": drafts,
           "index": index, "ivf": ivf}
    return res, ctx


def close_workload(ctx):
    import torch

    ctx["index"].close()
    if ctx["ivf"] is not None:
        ctx["ivf"].close()
    ctx.clear()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def config_summary(res):
    """The figures of one configuration's run kept in the headline line."""
    keep = ("ms_per_step", "value", "scan_ms", "filter_ms", "topk_ms", "verify_ms",
            "hbm_gbps", "hbm_read_ceiling_gbps", "roofline", "mfma", "retrieval_scan_gbps",
            "cpu_baseline")
    out = {k: res[k] for k in keep if k in res}
    out["queries_per_s"] = out.pop("value")
    c = res["config"]
    out["config"] = {k: c[k] for k in ("n", "d", "key_dtype", "n_queries", "k", "span", "vocab",
                                       "logits_dtype", "verify_candidates")}
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(its row-sharded design is not built); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_00021_amd import synth

    name = args.workload or synth.HEADLINE
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    K = args.steps
    res, ctx = run_workload(name, args, dev, K, args.warmup, graph=args.graph,
                            copy_probe_mib=args.copy_probe_mib)
    w = ctx["w"]
    if not args.no_sen and not w.proj:
        res["sen"] = sen_leg(args, w, ctx["ds"], ctx["q"], ctx["src_rows"], K, dev)
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host (cpu_baseline)")
        t0 = time.perf_counter()
        res["cpu_baseline"] = cpu_baseline(w, ctx["ds"], ctx["q"], ctx["logits"], ctx["drafts"],
                                           args.cpu_seconds)
        log(f"[bench] cpu_baseline took {time.perf_counter() - t0:.1f} s")
    close_workload(ctx)
    del ctx
    if args.workload is None and not args.no_configs:
        # Every other configuration once, on the same device, after the
        # headline (its own steps, fewer of them; no SEN leg; the oracle timed
        # on a smaller sample).
        res["configs"] = {}
        for cname in CONFIG_WORKLOADS:
            if cname == name:
                continue
            r, c = run_workload(cname, args, dev, min(K, 10), min(args.warmup, 2))
            if not args.no_cpu_baseline:
                # the oracle per query on this workload, a smaller sample
                r["cpu_baseline"] = cpu_baseline(c["w"], c["ds"], c["q"], c["logits"],
                                                 c["drafts"], args.config_cpu_seconds,
                                                 max_sample_bytes=2e9)
            close_workload(c)
            del c
            res["configs"][cname] = config_summary(r)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
