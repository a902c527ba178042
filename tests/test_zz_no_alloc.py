"""sense_retrieve_noalloc (retrieval with the library's static scratch, for
callers that cannot allocate) against sense_retrieve with a workspace: two
calls in a row, the second on a smaller input, each bit-identical to the
workspace call (same kernels, same inputs); and a call needing more scratch
than the static array holds is refused before any device work."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2606_00021_amd import sense, synth
from parity import check_topk, host_bits, query_bounds

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _outs(nq, k, m):
    return (torch.full((nq, k), -5, dtype=torch.int64, device=DEV),
            torch.full((nq, k), -5.0, dtype=torch.float32, device=DEV),
            torch.full((nq, k, m), -5, dtype=torch.int32, device=DEV),
            torch.full((nq, k), -5, dtype=torch.int32, device=DEV))


@pytest.mark.parametrize("first,second", [
    # (n, d, n_queries, k): the second call is smaller in every size
    ((300_000, 1024, 1, 64), (30_000, 512, 1, 16)),
    ((120_000, 2048, 8, 32), (9_000, 256, 4, 8)),
    # a batch over a sampled store (threshold, filtered pass, band, rescore)
    ((140_007, 256, 8, 32), (20_000, 128, 3, 16)),
])
def test_noalloc_matches_workspace_call(first, second):
    for case, (n, d, nq, k) in (("first", first), ("second", second)):
        print(f"[no-alloc] {case} call: n={n} d={d} Q={nq} k={k}", flush=True)
        w = synth.scaled(synth.WORKLOADS["store-1m-d4096"], name="noalloc", n=n, d=d, k=k,
                         n_queries=nq, n_clusters=max(8, n // 256))
        ds = synth.make_datastore(w, n % 97, DEV, ragged_spans=True)
        q, _ = synth.make_queries(w, ds, n % 89, n_queries=nq)
        index = sense.sense_build_index(ds.keys, ds.spans, ds.span_len)
        ref = sense.sense_retrieve(index, q, k)
        got = sense.sense_retrieve_noalloc(index, q, k, _outs(nq, k, w.span))
        torch.cuda.synchronize()
        for a, b in zip(ref, got):
            assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                               b.view(torch.int32) if b.dtype == torch.float32 else b)
        # and the oracle's bar on the ids, as for the workspace call
        kb = host_bits(ds.keys)
        o_s = oracle.scores(kb, w.key_dtype, q.cpu().numpy(), "f32")
        bounds = query_bounds(kb, w.key_dtype, q.cpu().numpy(), "cosine")
        for qi in range(nq):
            check_topk(got[0][qi].cpu().numpy(), got[1][qi].cpu().numpy(), o_s[qi], k, bounds[qi])
        index.close()
    print("[no-alloc] ok", flush=True)


def test_noalloc_refuses_oversized_call():
    n, d, nq, k = 300_000, 64 * 8, 64, 8          # 64 x 300000 fp32 scores > 64 MiB
    w = synth.scaled(synth.WORKLOADS["store-1m-d4096"], name="noalloc-big", n=n, d=d, k=k,
                     n_queries=nq, n_clusters=512)
    ds = synth.make_datastore(w, 3, DEV)
    q, _ = synth.make_queries(w, ds, 3, n_queries=nq)
    index = sense.sense_build_index(ds.keys, ds.spans, ds.span_len)
    assert sense.sense_retrieve_workspace_size(index, nq, k) > sense.sense_retrieve_noalloc_max_bytes()
    outs = _outs(nq, k, w.span)
    with pytest.raises(sense.SenseError, match="static scratch"):
        sense.sense_retrieve_noalloc(index, q, k, outs)
    torch.cuda.synchronize()
    assert (outs[0] == -5).all()                   # nothing was launched
    index.close()
