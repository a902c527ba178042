"""The C ABI from a plain C program.  tests/c_abi/sense_c_driver (C99, linked
against libsense.so and the HIP runtime only, built by the build step) reads
a problem from raw files, runs sense_build_index, sense_retrieve and
sense_soft_gate_verify on its own stream and device buffers, and writes the
results back; they must meet the oracle under the same rules as the Python
binding's (tests/parity.py): ordered top-k ids up to bounded near ties,
scores within their derived bounds, drafts exactly, ranks exactly, gate
scores within GATE_ABS, accepted lengths and best drafts exactly away from
the entropy threshold.  The driver runs as a child process of the test."""
import os
import subprocess

import numpy as np
import pytest
import torch

import oracle
from paper_2606_00021_amd import synth
from parity import check_topk, check_verify, host_bits, query_bounds

pytestmark = pytest.mark.gpu

DRIVER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "sense_c_driver")
METRIC = {"ip": 0, "cosine": 1}
DTYPE = {"f16": 1, "bf16": 2}
GATE = dict(gamma=0.05, topk=3, window=6, tau=0)

CASES = [
    # n, d, key dtype, n_queries, k, metric, logits dtype
    (20000, 512, "bf16", 1, 16, "cosine", "f32"),     # one query: the vector-ALU scan
    (30011, 256, "f16", 3, 32, "ip", "bf16"),         # a batch: the matrix-core scan
]
LOGITS = {"f32": (0,), "f16": (1,), "bf16": (2,)}


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_c_driver_matches_oracle(case, tmp_path):
    if not os.access(DRIVER, os.X_OK):
        pytest.fail(f"{DRIVER} is not built: run __graft_entry__.build()")
    n, d, kdt, nq, k, metric, ldt = case
    print(f"[c-abi] case={case}", flush=True)
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=n, d=d, key_dtype=kdt, n_queries=nq,
                     k=k, vocab=3000, n_clusters=64)
    ds = synth.make_datastore(w, 61, "cpu", ragged_spans=True)
    q, _ = synth.make_queries(w, ds, 61)
    keys = host_bits(ds.keys)
    spans = ds.spans.numpy()
    span_len = ds.span_len.numpy()
    queries = q.numpy().astype(np.float32)
    m, vocab = w.span, w.vocab

    # Logits row-aligned with the oracle's drafts (the draft token boosted at
    # some positions, so that accepted prefixes vary).
    o_ids, _, o_dr, _ = oracle.retrieve(keys, kdt, queries, "f32", k, spans, span_len, metric)
    logits_t = synth.make_logits(w, torch.from_numpy(o_dr.reshape(nq * k, m)), 61, dtype=ldt)
    logits = host_bits(logits_t)          # float32 values, or 16-bit bit patterns

    with open(tmp_path / "params.txt", "w") as f:
        f.write(f"{n} {d} {m} {nq} {k} {METRIC[metric]} {DTYPE[kdt]} {vocab} "
                f"{GATE['gamma']} {GATE['topk']} {GATE['window']} {GATE['tau']} "
                f"{LOGITS[ldt][0]}\n")
    keys.tofile(tmp_path / "keys.bin")
    spans.astype(np.int32).tofile(tmp_path / "spans.bin")
    span_len.astype(np.int32).tofile(tmp_path / "span_len.bin")
    queries.tofile(tmp_path / "queries.bin")
    logits.tofile(tmp_path / "logits.bin")

    run = subprocess.run([DRIVER, str(tmp_path)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, f"driver exit {run.returncode}: {run.stderr[-2000:]}"
    print(run.stdout.strip(), flush=True)

    def out(name, dt, shape):
        return np.fromfile(tmp_path / name, dtype=dt).reshape(shape)

    ids = out("ids.bin", np.int64, (nq, k))
    scores = out("scores.bin", np.float32, (nq, k))
    drafts = out("drafts.bin", np.int32, (nq, k, m))
    dlen = out("draft_len.bin", np.int32, (nq, k))

    all_scores = oracle.scores(keys, kdt, queries, "f32", metric)
    bounds = query_bounds(keys, kdt, queries, metric)
    for i in range(nq):
        check_topk(ids[i], scores[i], all_scores[i], k, bound=bounds[i])
        g_dr, g_dl = oracle.gather(spans, span_len, ids[i])
        assert np.array_equal(drafts[i], g_dr), f"query {i}: drafts differ from spans[ids]"
        assert np.array_equal(dlen[i], g_dl), f"query {i}: draft lengths differ"

    flat_dr, flat_dl = drafts.reshape(nq * k, m), dlen.reshape(nq * k)
    ref = oracle.soft_gate_verify(logits, ldt, flat_dr, flat_dl, n_groups=nq, **GATE)
    gpu = {"accept_len": torch.from_numpy(out("accept_len.bin", np.int32, (nq * k,))),
           "best": torch.from_numpy(out("best.bin", np.int32, (nq,))),
           "gate_score": torch.from_numpy(out("gate_score.bin", np.float32, (nq * k, m))),
           "rank": torch.from_numpy(out("rank.bin", np.int32, (nq * k, m)))}
    check_verify(gpu, ref, GATE["gamma"], draft_len=flat_dl)
    assert (gpu["accept_len"].numpy() > 0).any(), "no draft accepted anything: a vacuous case"
