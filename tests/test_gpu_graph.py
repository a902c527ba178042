"""The hot path is capturable in a HIP graph: the entry points allocate
nothing and record no memset, so a captured retrieve + verify step replays
to exactly the eager results.  Replays are interleaved with eager work and
synchronisations, and every replay is checked."""
import pytest
import torch

from paper_2606_00021_amd import sense, synth

pytestmark = pytest.mark.gpu


def test_graph_replay_matches_eager():
    dev = torch.device("cuda")
    w = synth.scaled(synth.WORKLOADS["store-1m-d4096"], n=30000, n_clusters=120)
    ds = synth.make_datastore(w, 21, dev)
    q, _ = synth.make_queries(w, ds, 21)
    index = sense.sense_build_index(ds.keys, ds.spans)
    k, m = w.k, w.span
    ws_r = torch.empty(sense.sense_retrieve_workspace_size(index, 1, k), dtype=torch.uint8, device=dev)
    outs = (torch.empty((1, k), dtype=torch.int64, device=dev),
            torch.empty((1, k), dtype=torch.float32, device=dev),
            torch.empty((1, k, m), dtype=torch.int32, device=dev),
            torch.empty((1, k), dtype=torch.int32, device=dev))
    sense.sense_retrieve(index, q, k, workspace=ws_r, out=outs)
    drafts, dlen = outs[2][0], outs[3][0]
    logits = synth.make_logits(w, drafts, 21)
    ws_v = torch.empty(sense.sense_soft_gate_verify_workspace_size(k, m, w.vocab),
                       dtype=torch.uint8, device=dev)
    out_v = {"accept_len": torch.empty(k, dtype=torch.int32, device=dev),
             "best": torch.empty(1, dtype=torch.int32, device=dev),
             "gate_score": torch.empty((k, m), dtype=torch.float32, device=dev)}

    def step(stream=None):
        sense.sense_retrieve(index, q, k, workspace=ws_r, out=outs, stream=stream)
        sense.sense_soft_gate_verify(logits, drafts, dlen, workspace=ws_v, out=out_v,
                                     stream=stream)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs] + [v.clone() for v in out_v.values()]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step(stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for _ in range(4):
        for t in list(outs) + list(out_v.values()):
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = list(outs) + list(out_v.values())
        for x, y in zip(got, ref):
            assert torch.equal(x, y)
        step()                                    # eager work between replays
        torch.cuda.synchronize()
    index.close()


@pytest.mark.parametrize("metric", ["cosine", "ip"])
def test_graph_replay_batched_sampled_retrieval(metric):
    """A batch over a store large enough for the sampled threshold (query
    split, sample pass and top-k, threshold, filtered pass with atomic
    overflow positions, survivors' top-k; for cosine also the band and its
    rescore) captured once and replayed: every replay equals the eager call."""
    dev = torch.device("cuda")
    w = synth.scaled(synth.WORKLOADS["13b-batched-4m-d5120"], n=140_007, d=256, k=64,
                     n_queries=16, n_clusters=600)
    ds = synth.make_datastore(w, 23, dev)
    q, _ = synth.make_queries(w, ds, 23)
    index = sense.sense_build_index(ds.keys, ds.spans, metric=metric)
    nq, k, m = w.n_queries, w.k, w.span
    ws = torch.empty(sense.sense_retrieve_workspace_size(index, nq, k), dtype=torch.uint8,
                     device=dev)
    outs = (torch.empty((nq, k), dtype=torch.int64, device=dev),
            torch.empty((nq, k), dtype=torch.float32, device=dev),
            torch.empty((nq, k, m), dtype=torch.int32, device=dev),
            torch.empty((nq, k), dtype=torch.int32, device=dev))

    def step(stream=None):
        sense.sense_retrieve(index, q, k, workspace=ws, out=outs, stream=stream)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step(stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for _ in range(4):
        for t in outs:
            t.zero_()
        ws.fill_(0xA5)                            # stale scratch must not matter
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for x, y in zip(outs, ref):
            assert torch.equal(x, y)
        step()
        torch.cuda.synchronize()
    index.close()


def test_concurrent_batched_retrievals_on_two_streams():
    """Two batched searches of one index on two streams with their own
    workspaces, enqueued so that they can overlap on the device, return
    exactly what each returns alone (the library keeps no global state
    between the kernels of a search)."""
    dev = torch.device("cuda")
    w = synth.scaled(synth.WORKLOADS["13b-batched-4m-d5120"], n=140_007, d=256, k=64,
                     n_queries=24, n_clusters=600)
    ds = synth.make_datastore(w, 29, dev)
    q, _ = synth.make_queries(w, ds, 29)
    index = sense.sense_build_index(ds.keys, ds.spans)
    qa, qb = q[:16].contiguous(), q[16:].contiguous()

    def bufs(nq):
        return (torch.empty((nq, w.k), dtype=torch.int64, device=dev),
                torch.empty((nq, w.k), dtype=torch.float32, device=dev),
                torch.empty((nq, w.k, w.span), dtype=torch.int32, device=dev),
                torch.empty((nq, w.k), dtype=torch.int32, device=dev))
    ws_a = torch.empty(sense.sense_retrieve_workspace_size(index, 16, w.k), dtype=torch.uint8,
                       device=dev)
    ws_b = torch.empty(sense.sense_retrieve_workspace_size(index, 8, w.k), dtype=torch.uint8,
                       device=dev)
    ref_a, ref_b = bufs(16), bufs(8)
    sense.sense_retrieve(index, qa, w.k, workspace=ws_a, out=ref_a)
    sense.sense_retrieve(index, qb, w.k, workspace=ws_b, out=ref_b)
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(3):
        out_a, out_b = bufs(16), bufs(8)
        torch.cuda.synchronize()
        sense.sense_retrieve(index, qa, w.k, workspace=ws_a, out=out_a, stream=sa)
        sense.sense_retrieve(index, qb, w.k, workspace=ws_b, out=out_b, stream=sb)
        torch.cuda.synchronize()
        for x, y in zip(out_a, ref_a):
            assert torch.equal(x, y)
        for x, y in zip(out_b, ref_b):
            assert torch.equal(x, y)
    index.close()
